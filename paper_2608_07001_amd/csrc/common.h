// Internal declarations shared by the HIP translation units of libgracekv.
// Target: gfx950 (CDNA4), wave64.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gracekv.h"

namespace gkv {

constexpr int NMAX = 128;        // longest slot (n_max); units hold at most 2*NMAX-1 nodes
constexpr int NODE_MAX = 2 * NMAX - 1;
constexpr int WMAX = 64;         // window queries
constexpr int DMAX = 128;        // head dim
constexpr int CAND_MAX = 18;     // prefix (or suffix) children per refinement: 17 cuts + extraction side

// Every size and hyperparameter a kernel needs, passed by value.
struct Dims {
  int L, G, H, d, hpg, W, n_seg, Dh, dtype;
  int r, J_cap;
  int64_t T, N_ctx, N_c, B_total, B_free;
  float lam_stab, lam_s, eps_seg, mad;
  int win[3];
  int n_min, n_max, n0;
  float lam_d, lam_n, c_cut;
  float lam_Z, lam_M, lam_kappa, beta_frac, eps;
  int k_curv;
  int rows;                      // relevance rows per (l, g): hpg * W
  int dp_serial;                 // segmentation DP: no warm-up guess, every chunk from the true state
  int uniform_slots;             // slots of n0 tokens instead of the DP partition (ablation)
  int pair_quotas;               // the auction with fixed per-(l, g) capacities (ablation)
  float lam_graph;               // weight of the multi-hop relevance in the token values
  int n_gl, gl[2];               // propagation layers of the multi-hop relevance
  int stage_times;               // record the stage clock's events (GRACEKV_FLAG_STAGE_TIMES)
  float alpha_floor;             // singleton floor share alpha (0: no floor)
  int64_t floor_cap;             // floor(alpha B_free): entries the floor may spend
};

// Typed views into the tree buffer (offsets come from gracekv_plan).
struct TreeView {
  int32_t* node_a;      // absolute start
  int32_t* node_n;      // length
  int32_t* node_child;  // first child (local index) or -1
  int32_t* node_parent; // parent (local index) or -1
  uint8_t* node_nch;
  uint8_t* node_kind;   // 0 leaf, 1 binary split, 2 extraction
  int32_t* node_cut;
  float* node_D;
  float* node_R;
  float* sp_U;          // Split op of node slot i
  uint64_t* sp_E;
  uint8_t* sp_cost;
  uint8_t* sp_exec;
  int32_t* unit_nn;     // nodes per unit
  float* unit_Ddrop;
  float* add_U;
  uint64_t* add_E;
  uint8_t* add_exec;
  float* tok_R;         // [LG][N_c] token values
  float* tok_A;         // [LG][N_c] mean normalised probe attention of each token
  float4* row_stats;    // [LG][rows] (m_V, Z_V, m_C, Z_C)
  float* probe_m;       // [LG][W]
  float* probe_ZC;      // [LG][W]
  float* lg_S;          // [LG]
  float* omega;         // [LG] normalised sensitivity
  int32_t* status;      // device status word
  int32_t* slots;       // [J_cap + 1] copy of the slot starts (then N_c)
  int32_t* nslots;      // [1] J
  uint64_t* theta;      // [2] pruned build: [0] lower bound of the auction cut, [1] root-split skip bound
  void* selstate;       // radix-select state of that bound
  int32_t* work;        // [L*G*J_cap][8] work items: unit, slot start, slot length, and the root's
                        // D, R (float bits), the sensitivity w (float bits), the Add key (two words)
  int32_t* wctr;        // [4] list length, next item
  void* proto;          // [unit_cap][2][d] root prototype (k~, v~) of each unit, cache dtype
  float* proto_logm;    // [unit_cap] log m_eff of the root
  void* kargs;          // device copy of the kernel arguments (Dims, then this view) for the
                        // kernels that read them through pointers
  const float* dhat;    // [N_c] multi-hop relevance to mix into the token values, or null
  // singleton floor (null without one)
  const uint8_t* fl_flag;   // [LG][N_c] 1: the token is an initial floor candidate of its (l, g)
  const uint8_t* fl_pre_add;  // [unit_cap] 1: the floor executed the unit's Add
  const uint8_t* fl_pre_sp;   // [node_cap] 1: the floor executed the node's Split
  const int64_t* fl_state;  // [8] B_floor first
  // level-by-level refinement (bf16): items [lv_cap][8] as in work (the slot
  // length word also holds the node's BFS index << 16, the Add key word the key
  // of the op that creates the node), results [lv_cap][12], two lists of the
  // units with nodes at the current depth, per unit (first, end, item base,
  // items) of that depth, and counters
  int32_t* lv_items;
  int32_t* lv_res;
  int32_t* lv_units;    // [2][unit_cap]
  int4* lv_state;       // [unit_cap]
  int32_t* lv_ctr;      // [16]
  int64_t lv_cap;
};
// bytes of the level region at the end of the tree buffer, and its item capacity
// (the nodes of one depth are disjoint, at least two tokens each: N_c / 2 per (l, g))
size_t level_region_bytes(int64_t LG, int64_t N_c, int64_t unit_cap);
int64_t level_capacity(int64_t LG, int64_t N_c);

// The singleton floor's region of the tree buffer (alpha_floor > 0).  Public
// part, each array 256-byte aligned in this order: int64 state[8] (B_floor,
// cap, total cost of the initial lists' paths, lists reduced, failure (l, g),
// failure index, cost realised before it), int32 cnt[LG] (initial list
// lengths), int32 keep[LG] (lengths after the proportional reduction), int32
// list[LG][N_c] (candidates in the floor's order), uint8 flag[LG][N_c], uint8
// pre_add[unit_cap], uint8 pre_sp[node_cap]; then scratch.
struct FloorView {
  int64_t* state;
  int32_t* cnt;
  int32_t* keep;
  int32_t* list;        // also the sort's first key/value buffer's values
  uint8_t* flag;
  uint8_t* pre_add;
  uint8_t* pre_sp;
  float* rbar;          // [N_c] mean token value over (l, g)
  uint32_t* keyA;       // [LG][N_c] sort keys (ping)
  uint32_t* keyB;       // [LG][N_c] sort keys (pong); then the tail's path costs
  int32_t* valB;        // [LG][N_c] sort values (pong); then the tail's unit ids
  int32_t* first_add;   // [unit_cap] first list index whose path holds the Add
  int32_t* first_sp;    // [node_cap] ... the Split
  int32_t* inc;         // [LG][N_c] incremental path cost of each candidate
  int64_t* lgsum;       // [LG] path cost of each (l, g)
  size_t bytes;
};
FloorView floor_view(void* base, const Dims& dm, int64_t unit_cap, int64_t node_cap);
hipError_t launch_floor_candidates(const Dims& dm, const TreeView& tv, const FloorView& fv, hipStream_t st);
hipError_t launch_floor_realise(const Dims& dm, const TreeView& tv, const FloorView& fv, hipStream_t st);

// Multi-hop relevance scratch (the build workspace when lambda_graph > 0).
struct MhView {
  float* dk;            // [N_c] seed score, then the current hop's scores
  float* dacc;          // [N_c] decayed sum of the hop scores
  float* dhat;          // [N_c] normalised sum
  int32_t* seeds;       // [64] current seeds
  float* wts;           // [64] their weights
  int32_t* ns;          // number of current seeds
  int32_t* used;        // [hops * 64] every seed so far
  int32_t* nused;
  float2* rstat;        // [groups][rows] (max, log2 partition sum) of each seed row
  float2* rpart;        // [chunks][groups][rows] their chunk partials
  float* dpart;         // [groups][row blocks][N_c] per-token partial sums
  uint64_t* cand;       // [blocks][64] seed candidates (score, position keys) of each block
  double* bsum;         // [blocks] score sum of each block
  size_t bytes;
};

// Refinement modes (the roots come from the root kernel): FULL refines every
// node; ROOT_SPLIT refines the root of units whose Add key reaches theta;
// CONTINUE refines every unrefined node whose creating op reaches theta.
// ROOT_FULL refines the root of every unit (the first level of the complete
// build).  For bf16 caches the roots are refined by their own kernel
// (launch_split_root) in ROOT_SPLIT and ROOT_FULL, and the next levels by the
// same kernel one depth at a time: LEVEL (pruned) and LEVEL_FULL (complete)
// take the nodes of one depth from a list and write one result per node, which
// the level pass then numbers in BFS order.
enum { BUILD_FULL = 0, BUILD_ROOT_SPLIT = 2, BUILD_CONTINUE = 3, BUILD_ROOT_FULL = 4, BUILD_LEVEL = 5,
       BUILD_LEVEL_FULL = 6 };
constexpr int LEVELS_MAX = 48;   // depths refined level by level; deeper nodes go to the per-unit kernel
constexpr int LEVELS_SPARSE = 12; // the same at a compression of 64x or more

// ---- gains, utilities and keys (shared by the build and score kernels so that
// both produce bit-identical keys) -------------------------------------------
// Add: Delta = w R(root) (D_drop - D); Split: Delta = w R(v) (D(v) - sum D(children)),
// cost |child| - 1; U = max(Delta, 0) / cost (App. A.5 eq:app_operation_gains,
// eq:app_operation_costs, eq:app_unit_utility; App. C.5 clamp at zero).
__device__ __forceinline__ float add_gain(float w, float R, float Ddrop, float D) { return w * R * (Ddrop - D); }
__device__ __forceinline__ float split_gain(float w, float R, float D, float sumD) { return w * R * (D - sumD); }
__device__ __forceinline__ float utility(float gain, int cost) {
  const float g = gain > 0.f ? gain : 0.f;
  return cost == 1 ? g : g / (float)cost;
}
// unique priority: larger U first, then the smaller id
__device__ __forceinline__ uint64_t op_key(float U, uint32_t id) {
  return ((uint64_t)__float_as_uint(U) << 32) | (uint64_t)(0xFFFFFFFFu - id);
}
// Upper bound of the key of a root's Split before the root is refined: the
// children's distortions are >= 0 and the cost is >= 1, and every rounding step
// of split_gain / utility is monotone, so the key the Split gets once its
// children are known (and its effective key) is <= this value, bit for bit.
__device__ __forceinline__ uint64_t root_split_key_bound(float w, float R, float D, uint32_t ord) {
  return op_key(utility(split_gain(w, R, D, 0.f), 1), ord * 256u + 1u);
}

// representative position of [x0, x1): round((x0 + x1 - 1) / 2), ties to even
__device__ __forceinline__ int round_half_even_mid(int x0, int x1) {
  const int s = x0 + x1 - 1;
  if ((s & 1) == 0) return s >> 1;
  const int h = s >> 1;
  return (h & 1) ? h + 1 : h;
}

Dims make_dims(const gracekv_config& c, const gracekv_plan& p);
size_t decode_ws_bytes(const Dims& dm, int P);
int decode_parts(const Dims& dm);
hipError_t launch_decode(const Dims& dm, const void* q, const int64_t* offsets, const void* K_out, const void* V_out,
                         const float* logm_out, const void* K, const void* V, float* out, void* ws, hipStream_t st);
// the same, with the partial states in the library's fixed device scratch
// (hipErrorInvalidValue when they exceed GRACEKV_DECODE_SCRATCH_BYTES)
hipError_t launch_decode_noalloc(const Dims& dm, const void* q, const int64_t* offsets, const void* K_out,
                                 const void* V_out, const float* logm_out, const void* K, const void* V, float* out,
                                 hipStream_t st);
// status word of the tree buffer: [0] latched fault bits, [1] the marker
// gracekv_build_trees writes first
constexpr int32_t STATUS_NUMERIC = 1, STATUS_PARTITION = 2, STATUS_CAPACITY = 4;
constexpr int32_t STATUS_BUILT = 0x4b56424c;
constexpr size_t KARGS_BYTES = 1024;      // tail of the tree buffer: Dims at 0, TreeView at 512
hipError_t launch_store_args(const Dims& dm, const TreeView& tv, hipStream_t st);
// bf16 caches with at most 8 query heads per KV head: the direct relevance s-hat
// of every token comes from its own pass (launch_token_relevance, after the row
// statistics) and the root kernel reads it from the token values.
inline bool token_relevance_pass(const Dims& dm) { return dm.dtype == GRACEKV_BF16 && dm.hpg <= 8 && dm.W <= 64; }
hipError_t launch_token_relevance(const Dims& dm, const void* K, const void* Q, const TreeView& tv, hipStream_t st);
size_t mh_bytes(const Dims& dm);
MhView mh_view(void* base, const Dims& dm);
hipError_t launch_multihop(const Dims& dm, const void* K, const void* Q, const void* Q_graph, const TreeView& tv,
                           void* mh_base, hipStream_t st);
TreeView make_view(void* base, const gracekv_plan& p);

// ---- device helpers -------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffff) ? 0x40 : 0));
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// element load as fp32 for the two storage types
__device__ __forceinline__ float ldf(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ldf(const uint16_t* p, int64_t i) { return bf16_to_f32(p[i]); }
__device__ __forceinline__ void stf(float* p, int64_t i, float v) { p[i] = v; }
__device__ __forceinline__ void stf(uint16_t* p, int64_t i, float v) { p[i] = f32_to_bf16_rne(v); }

// Workgroup barrier at the top of a loop whose previous iteration ended with
// LDS stores that the other waves read after it (a work-item index, a node
// table): the wave waits for its own LDS operations explicitly first.  The
// wait that the barrier's fence implies is not kept on such a loop back edge
// by the compiler, and without it a store may still be in flight, and be read
// stale by a wave on another SIMD, when the barrier opens.
__device__ __forceinline__ void sync_after_lds_stores() {
  __builtin_amdgcn_s_waitcnt(0xC07F);   // s_waitcnt lgkmcnt(0)
  __syncthreads();
}

// Workgroup barrier that orders LDS accesses only: unlike __syncthreads() it
// does not wait for the wave's global loads in flight.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Sum over the 16 lanes of each row (every lane gets it): lanes ^1, ^2 by
// quad permutes, then rotations by 4 and 8 within the row.
__device__ __forceinline__ float row_sum16(float v) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xf, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xf, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x124, 0xf, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xf, 0xf, false));
  return v;
}

// Last-workgroup hand-off without a device fence.  On this chip a device-scope
// fence writes back and invalidates the XCD's L2; where the only data the last
// workgroup reads are counters every workgroup updated with device-scope
// atomics, it suffices that each thread's atomics are performed before its
// workgroup takes a ticket (a wait on the vector-memory counter) and that the
// last workgroup reads the counters with device-coherent loads.
__device__ __forceinline__ void wait_vm() { __builtin_amdgcn_s_waitcnt(0x0F70); }   // s_waitcnt vmcnt(0)
template <typename T>
__device__ __forceinline__ T ld_agent(const T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Sum over the four lanes l % 16 + 16 k (one column of the four 16-lane rows),
// returned to all four: two row-swap permutations, no LDS traffic.  Every
// lane gets (r0 + r1) + (r2 + r3) in the same order.
__device__ __forceinline__ float col_sum4(float v) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}

// Wave all-reduces without LDS traffic: rotations by 8, 4, 2, 1 inside each
// 16-lane row (DPP), then the row swaps of col_sum4; every lane gets the result.
__device__ __forceinline__ float dpp_ror_f(float v, int ctrl_sel) {
  switch (ctrl_sel) {
    case 8: return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xf, 0xf, false));
    case 4: return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x124, 0xf, 0xf, false));
    case 2: return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x122, 0xf, 0xf, false));
    default: return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x121, 0xf, 0xf, false));
  }
}
__device__ __forceinline__ int dpp_ror_i(int v, int ctrl_sel) {
  switch (ctrl_sel) {
    case 8: return __builtin_amdgcn_update_dpp(0, v, 0x128, 0xf, 0xf, false);
    case 4: return __builtin_amdgcn_update_dpp(0, v, 0x124, 0xf, 0xf, false);
    case 2: return __builtin_amdgcn_update_dpp(0, v, 0x122, 0xf, 0xf, false);
    default: return __builtin_amdgcn_update_dpp(0, v, 0x121, 0xf, 0xf, false);
  }
}
// (value, index) with the larger value, ties to the smaller index, over the wave
__device__ __forceinline__ void wave_argmax(float& v, int& i) {
#pragma unroll
  for (int sh = 8; sh > 0; sh >>= 1) {
    const float v2 = dpp_ror_f(v, sh);
    const int i2 = dpp_ror_i(i, sh);
    if (v2 > v || (v2 == v && i2 < i)) { v = v2; i = i2; }
  }
  const auto pv = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  const auto pi = __builtin_amdgcn_permlane16_swap((uint32_t)i, (uint32_t)i, false, false);
  float a = __uint_as_float(pv[0]), b = __uint_as_float(pv[1]);
  int ia = (int)pi[0], ib = (int)pi[1];
  if (b > a || (b == a && ib < ia)) { a = b; ia = ib; }
  const auto qv = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(a), false, false);
  const auto qi = __builtin_amdgcn_permlane32_swap((uint32_t)ia, (uint32_t)ia, false, false);
  v = __uint_as_float(qv[0]); i = (int)qi[0];
  const float c = __uint_as_float(qv[1]);
  const int ic = (int)qi[1];
  if (c > v || (c == v && ic < i)) { v = c; i = ic; }
}
// minimum and maximum over the wave
__device__ __forceinline__ void wave_minmax(float& mn, float& mx) {
#pragma unroll
  for (int sh = 8; sh > 0; sh >>= 1) {
    mn = fminf(mn, dpp_ror_f(mn, sh));
    mx = fmaxf(mx, dpp_ror_f(mx, sh));
  }
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(mn), __float_as_uint(mn), false, false);
  const auto q = __builtin_amdgcn_permlane16_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
  mn = fminf(__uint_as_float(p[0]), __uint_as_float(p[1]));
  mx = fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1]));
  const auto p2 = __builtin_amdgcn_permlane32_swap(__float_as_uint(mn), __float_as_uint(mn), false, false);
  const auto q2 = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
  mn = fminf(__uint_as_float(p2[0]), __uint_as_float(p2[1]));
  mx = fmaxf(__uint_as_float(q2[0]), __uint_as_float(q2[1]));
}

// Sum over the wave, returned to every lane: 16-lane row sums by DPP, then the
// four row results read as scalars.
__device__ __forceinline__ float wave_sum_dpp(float v) {
  v = row_sum16(v);
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (r0 + r1) + (r2 + r3);
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// e^x as the hardware base-2 exponential (v_exp_f32, about 1 ulp) of
// x log2(e); the rounding of that product adds a relative error of about
// |x| 2^-24, the same order as the rounding already carried by x.
__device__ __forceinline__ float fexp(float x) { return __builtin_amdgcn_exp2f(x * 1.44269504088896341f); }

// Merge two (max, sum-of-exp) pairs: the sum is relative to its max.
__device__ __forceinline__ void lse_merge(float& m, float& z, float m2, float z2) {
  float mn = fmaxf(m, m2);
  if (mn == -INFINITY) { m = mn; z = 0.f; return; }
  z = z * expf(m - mn) + z2 * expf(m2 - mn);
  m = mn;
}

// ---- matrix cores ---------------------------------------------------------
// 16x16 output tile, C[i][j] += sum_k A[i][k] B[j][k].  Lane l holds
// C[4*(l/16) + r][l % 16] in acc[r].  For bf16 each step consumes 16 k: lane
// l supplies A[l%16][4*(l/16) .. +3] (same for B).  For fp32 each step
// consumes 4 k: lane l supplies A[l%16][l/16].
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// four bf16 packed two per 32-bit word (low half first) as an MFMA operand
__device__ __forceinline__ s16x4 pk4(uint32_t lo, uint32_t hi) {
  u32x2 v;
  v.x = lo;
  v.y = hi;
  return __builtin_bit_cast(s16x4, v);
}

__device__ __forceinline__ f32x4 mfma_bf16_16x16x16(s16x4 a, s16x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_f32_16x16x4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
// gfx950 16x16x32 bf16: lane l supplies A[l%16][8*(l/16) .. +7] and
// B[l%16][8*(l/16) .. +7] (eight bf16, low half of each 32-bit word first);
// output layout as above.  Twice the k of the 16x16x16 form per instruction.
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ s16x8 pk8(uint4 v) { return __builtin_bit_cast(s16x8, v); }
__device__ __forceinline__ f32x4 mfma_bf16_16x16x32(s16x8 a, s16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0,
                                                 0, 0);
}

// ---- launchers (each defined in its own translation unit) -----------------
hipError_t launch_rowstats(const Dims& dm, const void* K, const void* Q, const TreeView& tv, float4* partial,
                           hipStream_t st);
hipError_t launch_root(const Dims& dm, const void* K, const void* V, const void* Q, const float* cosT,
                       const float* sinT, const int32_t* slot_starts, const int32_t* n_slots, const TreeView& tv,
                       hipStream_t st);
int root_lds_bytes(const Dims& dm);
hipError_t launch_root_bf16(const Dims& dm, const void* K, const void* V, const void* Q, const float* cosT,
                            const float* sinT, const int32_t* slot_starts, const int32_t* n_slots, const TreeView& tv,
                            hipStream_t st);
int root_bf16_lds_bytes(int d);
// listed: the work list is already made (by the level passes); otherwise the
// units with nodes to refine are listed first
hipError_t launch_build(const Dims& dm, int lds_bytes, int mode, const void* K, const void* V, const void* Q,
                        const float* cosT, const float* sinT, const int32_t* slot_starts, const int32_t* n_slots,
                        const float* kappa, const TreeView& tv, hipStream_t st, bool listed = false);
hipError_t launch_omega(const Dims& dm, const float* omega_raw, const TreeView& tv, hipStream_t st);
// rank: B_free - 1 (the cut) or B_free (the skip bound, also stored in theta[1])
hipError_t launch_theta(const Dims& dm, const TreeView& tv, hipStream_t st, bool skip_bound);
size_t selstate_bytes(const Dims& dm);
hipError_t launch_score(const Dims& dm, const float* omega_raw, const TreeView& tv, hipStream_t st);
hipError_t launch_select(const Dims& dm, const TreeView& tv, int64_t* b_used, void* ws, hipStream_t st);
hipError_t launch_pack(const Dims& dm, const void* K, const void* V, const float* cosT, const float* sinT,
                       const TreeView& tv, int64_t* offsets, int64_t* counts, void* K_out, void* V_out,
                       int32_t* pos_out, float* logm_out, void* ws, hipStream_t st);
hipError_t launch_segment(const Dims& dm, const void* hidden, const float* surprisal, float* kappa, float* bscore,
                          int32_t* slot_starts, int32_t* n_slots, void* ws, hipStream_t st);
size_t segment_ws_bytes(const Dims& dm);
size_t select_ws_bytes(const Dims& dm);
size_t pack_ws_bytes(const Dims& dm);
int rowstats_chunks(const Dims& dm);
int build_lds_bytes(const Dims& dm);
int split_root_lds_bytes(int d);
hipError_t launch_split_root(const Dims& dm, int mode, const void* K, const void* V, const void* Q, const float* cosT,
                             const float* sinT, const int32_t* slot_starts, const int32_t* n_slots, const float* kappa,
                             const TreeView& tv, int grid, hipStream_t st);
// the levels below the roots (bf16): LEVELS_MAX (or LEVELS_SPARSE) rounds of the split kernel over
// one depth's list and the level pass; full: the complete build
hipError_t launch_levels(const Dims& dm, bool full, const void* K, const void* V, const void* Q, const float* cosT,
                         const float* sinT, const int32_t* slot_starts, const int32_t* n_slots, const float* kappa,
                         const TreeView& tv, int grid, hipStream_t st);
hipError_t launch_levels_bf16(const Dims& dm, bool full, const void* K, const void* V, const void* Q,
                              const float* cosT, const float* sinT, const int32_t* slot_starts,
                              const int32_t* n_slots, const float* kappa, const TreeView& tv, hipStream_t st);
hipError_t selftest_mfma(int which, float* out, hipStream_t st);

// Stage clock (GRACEKV_FLAG_STAGE_TIMES; stage ids GRACEKV_STAGE_*): clock_begin
// records the first event of a pair on the stream and returns its handle (-1
// when the clock is off or no event could be had); clock_end records the second.
int clock_begin(const Dims& dm, int stage, hipStream_t st);
void clock_end(int handle, hipStream_t st);

}  // namespace gkv
