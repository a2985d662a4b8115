/*
 * gracekv.h -- C ABI of the MI355X (gfx950) implementation of GraceKV's
 * one-shot, post-prefill KV-cache compression (arXiv 2608.07001).
 *
 * The path has five calls, run in this order on one HIP stream:
 *   gracekv_segment      curvature-guided slot partition      (App. B.2-B.3)
 *   gracekv_build_trees  direct relevance + prototype trees    (App. A.3-A.4)
 *   gracekv_score        Add / Split gains, utilities, keys    (App. A.5 eq:app_operation_gains..eq:app_unit_utility)
 *   gracekv_select       global budgeted greedy auction        (App. A.5 Stage II, App. C.3)
 *   gracekv_pack         ragged compressed cache               (App. A.5 "Frontier updates and physical packing")
 *
 * Conventions shared by every call
 *   - Positions are absolute.  The sequence is the context [0, N_ctx) followed
 *     by a question suffix of W tokens [N_ctx, T), T = N_ctx + W (no prompt
 *     prefix, c_s = 0).  The W window queries sit at the suffix positions and
 *     are both the direct-relevance probes and the distortion probes.
 *   - The recent window r and the budgets follow eq:app_total_budget,
 *     eq:app_compressible_context and eq:app_free_budget with the singleton
 *     floor disabled (alpha = 0, the paper's "w/o SF" setting).  The token
 *     values are the direct relevance alone when lambda_graph = 0 (the "w/o MH"
 *     setting) and mix in the multi-hop relevance when lambda_graph > 0
 *     (gracekv_build_trees).  Compressible context C = [0, N_c), N_c = N_ctx - r.
 *   - Every pointer argument except `cfg`, `plan` and host-side outputs is a
 *     DEVICE pointer owned by the caller; the library never allocates, frees or
 *     synchronises device memory (gracekv_plan reports every size).  All device
 *     buffers must be 16-byte aligned.
 *   - `stream` is a hipStream_t passed as void*; kernels are only enqueued.
 *   - Layouts are row-major:  K, V [L][G][T][d];  Q [L][H][W][d];
 *     hidden [n_seg][T][D_hidden];  rope_cos/rope_sin [T][d/2] fp32 (rotate-half
 *     RoPE: the pair (i, i + d/2) turns by the angle p theta_i of row p, so the
 *     turn from position p to position p' is that of row |p' - p| with the sine
 *     negated when p' < p; the library uses both forms);  K/V/Q/hidden are all
 *     of cfg->dtype.  Query head h belongs to KV head h / (H/G).
 *   - Errors: argument errors are detected on the host before anything is
 *     enqueued and return GRACEKV_ERR_INVALID_ARG / _UNSUPPORTED / _BUDGET /
 *     _WORKSPACE.  A failed launch returns GRACEKV_ERR_HIP.  Faults found on
 *     the device (a non-finite gain, a malformed slot partition, a packed
 *     cache over capacity) are latched in the status word inside the tree
 *     buffer and returned by gracekv_check.  gracekv_build_trees clears the
 *     word and marks the buffer as built before any kernel can latch a fault.
 */
#ifndef GRACEKV_H
#define GRACEKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GRACEKV_OK = 0,
  GRACEKV_ERR_INVALID_ARG = -1,
  GRACEKV_ERR_UNSUPPORTED = -2,
  GRACEKV_ERR_BUDGET = -3,
  GRACEKV_ERR_WORKSPACE = -4,
  GRACEKV_ERR_HIP = -5,
  GRACEKV_ERR_NUMERIC = -6,    /* a non-finite gain or utility (device) */
  GRACEKV_ERR_STATE = -7,      /* the tree buffer holds no build (gracekv_check) */
  GRACEKV_ERR_PARTITION = -8,  /* slot partition malformed: J outside [1, J_cap] (device) */
  GRACEKV_ERR_CAPACITY = -9    /* the packed cache would exceed B_total entries (device) */
} gracekv_status;

typedef enum { GRACEKV_F32 = 0, GRACEKV_BF16 = 1 } gracekv_dtype;

/* Version of this interface (structures and signatures).  A binding must
 * refuse a library whose gracekv_abi_version() differs from the value it was
 * written for: argument lists shift silently across versions. */
#define GRACEKV_ABI_VERSION 11

/* Shapes and hyperparameters.  gracekv_default_config fills the paper's
 * defaults (App. A and B); the caller then sets the shape fields. */
typedef struct {
  int32_t L, G, H, d;      /* layers, KV heads, query heads, head dim: 64 or 128 (fp32 data: 64) */
  int32_t n_seg;           /* hidden-state slabs (|L_seg|, eq:app_seg_layers), 1..8 */
  int32_t D_hidden;        /* hidden size of each slab (a multiple of 8) */
  int32_t W;               /* window queries (1..64) */
  int32_t dtype;           /* gracekv_dtype of K, V, Q and hidden */
  int64_t N_ctx;           /* context length */
  double x;                /* compression ratio x >= 1 (eq:app_total_budget) */
  int32_t r_default, r_min;                  /* recent window 32, minimum 4 (App. A.1) */
  float lam_stab, lam_s, eps_seg, mad_factor; /* 0.25, 0.15, 1e-6, 1.4826 (App. B.2) */
  int32_t win[3];                            /* curvature windows {4, 8, 16} */
  int32_t n_min, n_max, n0;                  /* 16, 128, 64 (eq:app_slot_length_defaults) */
  float lam_d, lam_n, c_cut;                 /* 0.25, 0.10, 1.0 (eq:app_segmentation_defaults) */
  float lam_Z, lam_M;                        /* 0.25, 0.75 (eq:app_probe_distortion) */
  int32_t k_curv;                            /* 16 curvature split candidates (0: midpoint only) */
  float lam_kappa, beta_frac, eps;           /* 0.05, 0.1, 1e-6 */
  float lambda_graph;                        /* multi-hop weight in [0, 1]: 0 (direct relevance
                                                only) or e.g. 0.3 (App. A.4 eq:app_bottom_up_value) */
  double alpha_floor;                        /* singleton floor share in [0, 1]: 0 (no floor) or
                                                e.g. 0.6 (App. A.5 Stage I, eq:app_floor_cap); with a
                                                floor the build is complete (no GRACEKV_FLAG_PRUNE,
                                                no GRACEKV_FLAG_PAIR_QUOTAS) */
  int32_t flags;                             /* GRACEKV_FLAG_* below */
} gracekv_config;

/* Budget-aware pruning of the tree build (output unchanged; see gracekv_build_trees). */
#define GRACEKV_FLAG_PRUNE 1
/* Segmentation DP without the chunk-parallel guess: every chunk of the
 * recurrence is run from the true state, one after the other (output
 * unchanged, slower; see gracekv_segment). */
#define GRACEKV_FLAG_DP_SERIAL 2
/* Uniform slots of n0 tokens (the last one shorter) instead of the curvature-
 * guided partition: the segmentation half of the paper's "w/o Curv.
 * Segmentation" ablation (App. C.4); kappa and b are still computed.  With
 * k_curv = 0 and lam_kappa = 0 the tree refinement is that ablation's too
 * (the interval midpoint as the only binary candidate, no curvature reward).
 * Needs n_min <= n0 <= n_max. */
#define GRACEKV_FLAG_UNIFORM_SLOTS 4
/* Fixed per-(l, g) capacities instead of the shared budget: the paper's "w/o
 * Global Allocation" ablation (App. C.3).  Pair i = l*G + g gets
 * floor(B_free / (L G)) entries, plus one for i < B_free mod (L G), and runs
 * the auction on its own ops; budget it leaves unused is not used elsewhere.
 * Not with GRACEKV_FLAG_PRUNE (whose bounds belong to the shared auction). */
#define GRACEKV_FLAG_PAIR_QUOTAS 8
/* gracekv_build_trees skips the relevance row statistics: the caller has run
 * gracekv_relevance_stats on the same tree buffer, completed before this call
 * starts (same stream, or joined with an event). */
#define GRACEKV_FLAG_STATS_READY 16
/* Stage clock: the calls record a pair of HIP events on their stream around
 * the main kernels of each stage (GRACEKV_STAGE_* below); gracekv_stage_times
 * reads them.  Output unchanged. */
#define GRACEKV_FLAG_STAGE_TIMES 32

/* Stages timed with GRACEKV_FLAG_STAGE_TIMES: the kernels between the two events. */
#define GRACEKV_STAGE_SEGMENT 0          /* every kernel of gracekv_segment */
#define GRACEKV_STAGE_ROWSTATS 1         /* relevance row statistics (pass 1), both kernels */
#define GRACEKV_STAGE_TOKEN_RELEVANCE 2  /* token relevance (pass 2, bf16 caches) */
#define GRACEKV_STAGE_ROOT 3             /* root evaluation of every unit */
#define GRACEKV_STAGE_ROOT_SPLIT 4       /* refinement of the roots (bf16: its own kernel) */
#define GRACEKV_STAGE_REFINE 5           /* refinement below the roots (pruned build) or of every
                                            node (complete fp32 build) */
#define GRACEKV_STAGE_PACK 6             /* gracekv_pack's emitting kernel */
#define GRACEKV_STAGE_FLOOR_CANDIDATES 7 /* singleton floor: scores, sorted candidate lists */
#define GRACEKV_STAGE_FLOOR_REALISE 8    /* singleton floor: path costs, reduction, realisation */
#define GRACEKV_N_STAGES 9

/* Sizes derived from a config (host only). */
typedef struct {
  int64_t T, N_c, B_total, B_free;
  int32_t r;
  int32_t J_cap;           /* slot capacity floor(N_c / n_min) + 1 */
  int64_t unit_cap;        /* L * G * J_cap */
  int64_t node_cap;        /* L * G * 2 * N_c node-table entries */
  size_t seg_ws_bytes;     /* workspace of gracekv_segment */
  size_t tree_bytes;       /* the tree buffer shared by build/score/select/pack */
  size_t sel_ws_bytes;     /* workspace of gracekv_select */
  size_t pack_ws_bytes;    /* workspace of gracekv_pack */
  /* byte offsets of the tree buffer's arrays (see gracekv_build_trees) */
  size_t off_node_a, off_node_n, off_node_child, off_node_parent, off_node_nch,
         off_node_kind, off_node_cut, off_node_D, off_node_R,
         off_sp_U, off_sp_E, off_sp_cost, off_sp_exec,
         off_unit_nn, off_unit_Ddrop, off_add_U, off_add_E, off_add_exec,
         off_tok_R, off_tok_A, off_row_stats, off_probe_m, off_probe_ZC, off_lg_S,
         off_omega, off_status, off_slots, off_nslots, off_partial, off_theta, off_selstate,
         off_work, off_wctr, off_proto, off_proto_logm,
         off_floor;        /* the singleton floor's region (alpha_floor > 0; see gracekv_select) */
  int32_t build_lds_bytes; /* dynamic LDS of the tree-build kernel */
  size_t build_ws_bytes;   /* workspace of gracekv_build_trees: 0 unless lambda_graph > 0 */
} gracekv_plan;

/* GRACEKV_ABI_VERSION of the compiled library. */
int32_t gracekv_abi_version(void);

/* Paper defaults (App. A, App. B): see the field comments above. */
gracekv_status gracekv_default_config(gracekv_config* cfg);

/* Validates cfg and fills plan.  Returns GRACEKV_ERR_BUDGET when the budget
 * cannot hold a recent window of r_min entries per (layer, KV head)
 * (App. A.1), GRACEKV_ERR_INVALID_ARG for lambda_graph outside [0, 1],
 * or alpha_floor outside [0, 1], GRACEKV_ERR_UNSUPPORTED for alpha_floor > 0
 * with GRACEKV_FLAG_PRUNE or GRACEKV_FLAG_PAIR_QUOTAS, lambda_graph > 0 with
 * H / G > 8, or shapes outside the documented limits. */
gracekv_status gracekv_plan_sizes(const gracekv_config* cfg, gracekv_plan* plan);

/* Human-readable name of a status. */
const char* gracekv_status_string(gracekv_status s);

/* Synchronises `stream` and reads the status word of the tree buffer.
 * Returns GRACEKV_ERR_STATE when no gracekv_build_trees call has been enqueued
 * on the buffer (a buffer is recognised as built by a marker that call writes
 * first; a caller that allocates the buffer should zero its first use, which
 * the Python binding does), else the first latched fault in this order:
 * GRACEKV_ERR_NUMERIC (a non-finite gain or utility in gracekv_score),
 * GRACEKV_ERR_PARTITION (gracekv_build_trees found J outside [1, J_cap]),
 * GRACEKV_ERR_CAPACITY (gracekv_pack found more frontier entries than
 * B_total), else GRACEKV_OK.  The word covers the calls since the last
 * gracekv_build_trees on the buffer. */
gracekv_status gracekv_check(const gracekv_config* cfg, void* trees, void* stream);

/* Stage clock (measurement, no part of the method).  Waits for every event
 * pair the calls with GRACEKV_FLAG_STAGE_TIMES recorded since the previous
 * gracekv_stage_times call (on any device and stream of this process), adds
 * the elapsed times per stage and forgets the pairs.
 *   total_ms   [GRACEKV_N_STAGES] fp32 host out: summed milliseconds per stage
 *   launches   [GRACEKV_N_STAGES] int32 host out: event pairs per stage
 * The events are created on first use and reused (they are not device
 * memory).  Returns GRACEKV_ERR_HIP if an event cannot be read. */
gracekv_status gracekv_stage_times(float* total_ms, int32_t* launches);

/* Curvature-guided slot segmentation (App. B.2 eq:app_hidden_normalization ..
 * eq:app_boundary_score; App. B.3 eq:app_adjacent_difference ..
 * eq:app_terminal_predecessor).
 *   hidden     [n_seg][T][D_hidden] (cfg->dtype), the slabs at the segmentation depths
 *   surprisal  [T] fp32, surprisal of each token (position 0 holds 0)
 *   kappa      [T] fp32 out: stabilized curvature (eq:app_stabilized_curvature)
 *   bscore     [T] fp32 out: boundary score b_i (eq:app_boundary_score)
 *   slot_starts [J_cap + 1] int32 out: slot starts a_1 = 0 < ... < a_J, then N_c
 *   n_slots    [1] int32 out: J
 *   ws         workspace of plan.seg_ws_bytes bytes
 * The recurrence runs on slot scores rounded once to a common fixed-point grid
 * (a power-of-two step chosen from the largest |score|, finer than 1e-12 for
 * scores of order one), so its additions are exact; chunks of 1024 ends are
 * solved in parallel from a guessed state and accepted only where that is
 * provably exact, the rest is recomputed (GRACEKV_FLAG_DP_SERIAL recomputes
 * all of them).  Ties go to the smallest slot start. */
gracekv_status gracekv_segment(const gracekv_config* cfg, const void* hidden, const float* surprisal,
                               float* kappa, float* bscore, int32_t* slot_starts, int32_t* n_slots,
                               void* ws, size_t ws_bytes, void* stream);

/* Direct relevance and one prototype tree per (layer, KV head, slot) unit
 * (App. A.3 eq:app_rope_prototype .. eq:app_split_choice; App. A.4
 * eq:app_attention_probability, eq:app_direct_relevance, eq:app_bottom_up_value;
 * App. B.4 eq:app_tree_split_candidates).
 *   K, V       [L][G][T][d], Q [L][H][W][d] (cfg->dtype)
 *   rope_cos/rope_sin [T][d/2] fp32
 *   slot_starts, n_slots, kappa: outputs of gracekv_segment (or caller-made)
 *   omega_raw  [L][G] fp32 raw sensitivity (or NULL for ones); read only with
 *              GRACEKV_FLAG_PRUNE, which needs the gains to bound the auction
 *   trees      the tree buffer (plan.tree_bytes).  Unit u = (l*G + g)*J_cap + j
 *              owns node slots [(l*G+g)*2*N_c + 2*a_j, ... + 2*n_j); nodes are in
 *              BFS order (root first; children of a node are contiguous, left to
 *              right).  Node arrays: start (int32, absolute), length (int32),
 *              first child (int32 local index, -1 for a leaf), parent (int32 local,
 *              -1 for the root), #children (uint8), kind (uint8: 0 leaf, 1 binary,
 *              2 extraction), cut (int32: xi or the extracted token), D and R (fp32).
 *              Per unit: node count (int32), D_drop of the root (fp32).  Token
 *              values R^tok [L*G][N_c] fp32; per (l,g) row statistics of the
 *              relevance softmax and the probe shifts m_q and Z_q(C); a copy of
 *              the slot partition (read by score, select and pack); per unit the
 *              root prototype (k~ then v~, d values each, rounded to cfg->dtype)
 *              and its log m_eff (fp32), which pack copies for a root on the
 *              frontier; the last 1024 bytes hold a device copy of the kernel
 *              arguments, rewritten in stream order by every call.
 *   Q_graph    [n_graph][H][T][d] (cfg->dtype) post-RoPE queries of every
 *              position at the propagation layers floor(0.50 L) and
 *              floor(0.75 L) (each capped at L - 1, a repeat dropped, so n_graph
 *              is 1 or 2); read only when lambda_graph > 0 (else pass NULL)
 *   ws         plan.build_ws_bytes of workspace when lambda_graph > 0 (NULL, 0
 *              otherwise); its contents need no initialisation
 * Multi-hop relevance (lambda_graph > 0; App. A.4 eq:app_global_seed_score,
 * eq:app_hop_propagation, eq:app_diffused_relevance, eq:app_bottom_up_value):
 * the seed score is the mean of s-hat over every (l, g); seeds are taken in
 * descending score (ties to the smaller position) until their cumulative share
 * of the total reaches 0.9 (the one reaching it included), at most 64, weighted
 * by their normalised scores; hop k sums, over the propagation layers, KV
 * heads, their query heads and the seeds u, w_u times the causal attention
 * probability of the query at u (range [0, u]) on each token of C; the scores
 * at the current and earlier seeds are then zeroed and the next hop seeds from
 * them; d = d^(1) + 0.5 d^(2), d-hat = d / (sum_C d + eps), and every token
 * value becomes (1 - lambda_graph) s-hat + lambda_graph d-hat.  Needs
 * H / G <= 8.
 * The direct relevance s-hat of every token: for bf16 caches with H / G <= 8
 * a pass of its own writes it into the token values before the roots are
 * evaluated (the root pass then reads it and mixes in d-hat); otherwise the
 * root pass computes it (and, with lambda_graph > 0, runs once without and once
 * with the mix).
 * With GRACEKV_FLAG_PRUNE the trees are built only as deep as the auction can
 * reach: every unit's root is evaluated; a cost-weighted radix pass over the ops
 * known so far gives theta_lb, the (B_free-1)-th largest effective key among
 * them, which bounds the final cut from below (more ops only raise it and
 * known effective keys never change); a node is refined only if the op that
 * creates it has E >= theta_lb.  A node that is not refined could be neither
 * split nor on the final frontier, so score, select and pack give the same
 * result as the full build.
 * For bf16 caches the nodes below the roots are refined one depth at a time
 * (all units at once) for up to 48 depths, or 12 where 64 B_total <= L G
 * N_ctx (a compression of 64x or more), the rest unit by unit, in the pruned
 * and the complete build alike; the environment variable GRACEKV_LEVELS
 * (0 .. 48, read at each call) sets that number instead, for tests of the
 * unit-by-unit continuation; the result does not depend on it beyond fp32
 * rounding of the distortions. */
gracekv_status gracekv_build_trees(const gracekv_config* cfg, const void* K, const void* V, const void* Q,
                                   const void* Q_graph, const float* rope_cos, const float* rope_sin,
                                   const int32_t* slot_starts, const int32_t* n_slots, const float* kappa,
                                   const float* omega_raw, void* trees, void* ws, size_t ws_bytes, void* stream);

/* Gains, utilities and priority keys (App. A.5 eq:app_operation_gains,
 * eq:app_operation_costs, eq:app_unit_utility; eq:app_head_sensitivity).
 *   omega_raw  [L][G] fp32 raw sensitivity, or NULL for all ones.
 * For every op: Delta+ = max(Delta, 0), U = Delta+ / c, composite key
 * k = (bits(U) << 32) | (2^32 - 1 - id) with id = unit ordinal * 256 + local
 * index (Add 0, Split(node i) 1 + i) and unit ordinal (l*G + g)*J + j, and the
 * effective key E = min(k, E(parent op)). */
gracekv_status gracekv_score(const gracekv_config* cfg, const float* omega_raw, void* trees, void* stream);

/* The budgeted greedy auction of App. A.5 / App. C.3, computed exactly: a
 * cost-weighted radix select over E finds the cut; ops above it execute, the
 * single group at the cut is resolved by the literal queue rule, and a
 * remaining single budget unit buys the best available cost-1 op.
 *   b_used     [1] int64 out: budget spent by the auction
 *   ws         workspace of plan.sel_ws_bytes bytes */
gracekv_status gracekv_select(const gracekv_config* cfg, void* trees, int64_t* b_used, void* ws, size_t ws_bytes,
                              void* stream);

/* Ragged compressed cache (App. A.5 "Frontier updates and physical packing").
 * Per (l, g), in ascending position: every frontier node (singleton: original
 * K/V, its position, log m = 0; other: prototype k~, v~ rounded to cfg->dtype,
 * representative position p_v, log m_eff), then the r recent-window tokens.
 *   offsets    [L*G + 1] int64 out (CSR), counts [L*G] int64 out
 *   K_out, V_out [B_total][d] (cfg->dtype), pos_out [B_total] int32,
 *   logm_out [B_total] fp32
 *   ws         workspace of plan.pack_ws_bytes bytes */
gracekv_status gracekv_pack(const gracekv_config* cfg, const void* K, const void* V,
                            const float* rope_cos, const float* rope_sin, void* trees,
                            int64_t* offsets, int64_t* counts, void* K_out, void* V_out,
                            int32_t* pos_out, float* logm_out, void* ws, size_t ws_bytes, void* stream);

/* Pass 1 of the direct relevance (App. A.4 eq:app_attention_probability,
 * eq:app_direct_relevance) on its own: per (l, g) and probe row the maximum
 * and partition sum of the logits over the visible range and over C, the
 * normaliser S_{l,g} and the probe shifts m_q, Z_q(C), written into the tree
 * buffer (plan.tree_bytes).  It needs neither the hidden states nor the slot
 * partition, so it can run on a second stream while gracekv_segment runs;
 * gracekv_build_trees then takes GRACEKV_FLAG_STATS_READY.  (Pass 2, s-hat of
 * every token, runs inside gracekv_build_trees: for bf16 caches with
 * H / G <= 8 as a pass of its own before the roots, else inside the roots.)
 *   K [L][G][T][d], Q [L][H][W][d] (cfg->dtype), 16-byte aligned; trees as in
 *   gracekv_build_trees.  Enqueued on stream, nothing allocated. */
gracekv_status gracekv_relevance_stats(const gracekv_config* cfg, const void* K, const void* Q, void* trees,
                                       void* stream);

/* Workspace of gracekv_decode_attention for this configuration (bytes). */
gracekv_status gracekv_decode_ws_bytes(const gracekv_config* cfg, size_t* ws_bytes);

/* Decode-time attention over the packed cache (App. A.3 eq:app_decode_logit;
 * App. A.5 "Frontier updates and physical packing": every entry stores k~, v~
 * and log m_eff, and attention at decode time adds log m_eff to the logit).
 * For every layer l and query head h, with KV head g = h / (H / G), the query
 * q[l][h] attends to the packed entries offsets[l*G+g] .. offsets[l*G+g+1] - 1
 * with logits q.k_i / sqrt(d) + logm_out[i], and to the window rows
 * N_ctx .. T-1 of K[l][g], V[l][g] (kept exactly, log m_eff = 0); out[l][h]
 * is the softmax-weighted mean of the values (fp32).
 *   q          [L][H][d] (cfg->dtype), already rotated to its position
 *   offsets    [L*G + 1] int64, K_out / V_out [B_total][d] (cfg->dtype),
 *              logm_out [B_total] fp32: the outputs of gracekv_pack (device);
 *              offsets outside [0, B_total] are clamped into it, a decreasing
 *              pair gives an empty row
 *   K, V       [L][G][T][d] (cfg->dtype): only the window rows are read
 *   out        [L][H][d] fp32 (device), written
 *   ws         workspace of gracekv_decode_ws_bytes bytes (partial softmax
 *              states of the split over entries), 16-byte aligned; calls that
 *              overlap on one workspace race
 * Returns GRACEKV_ERR_INVALID_ARG for null or misaligned pointers and
 * GRACEKV_ERR_WORKSPACE for a short workspace; enqueued on stream, nothing is
 * allocated or synchronised. */
gracekv_status gracekv_decode_attention(const gracekv_config* cfg, const void* q, const int64_t* offsets,
                                        const void* K_out, const void* V_out, const float* logm_out,
                                        const void* K, const void* V, float* out, void* ws, size_t ws_bytes,
                                        void* stream);

/* Size of the fixed device scratch of gracekv_decode_attention_noalloc (bytes). */
#define GRACEKV_DECODE_SCRATCH_BYTES (64u << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * computation as gracekv_decode_attention, with the same arguments except the
 * workspace, whose partial softmax states go to a fixed scratch array of
 * GRACEKV_DECODE_SCRATCH_BYTES inside the library instead.  Each GPU holds
 * its own copy of that array from the first call on it until the process
 * ends; the library locates it once per device (the device current at the
 * call) and never allocates, frees or synchronises.  Every partial state a
 * call reads is written by the same call, so nothing needs clearing.  Calls
 * that overlap on one GPU (on different streams, or from several host
 * threads) share the array and race: serialise them.
 * Returns GRACEKV_ERR_WORKSPACE, before anything is enqueued, when the partial
 * states of cfg (gracekv_decode_ws_bytes) exceed GRACEKV_DECODE_SCRATCH_BYTES
 * (the 8B-shaped caches fit at every ratio, the 70B-shaped 32K share from
 * about 11x), and the errors of gracekv_decode_attention
 * otherwise. */
gracekv_status gracekv_decode_attention_noalloc(const gracekv_config* cfg, const void* q, const int64_t* offsets,
                                                const void* K_out, const void* V_out, const float* logm_out,
                                                const void* K, const void* V, float* out, void* stream);

/* Layout check of the cross-lane instructions used by the kernels: computes
 * a 16x16 product from fixed inputs with the fp32 16x16x4 (which = 0), the
 * bf16 16x16x16 (which = 1) or the bf16 16x16x32 (which = 2) matrix
 * instruction, or (which = 3) the sum of lane + 1 over the four lanes
 * l % 16 + 16 k of a wave (out[0..63], the rest 0), into the caller's device
 * buffer out[256] (fp32, row-major 16x16).  Enqueued on stream; nothing is
 * allocated or synchronised. */
gracekv_status gracekv_selftest_mfma(int32_t which, float* out, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* GRACEKV_H */
