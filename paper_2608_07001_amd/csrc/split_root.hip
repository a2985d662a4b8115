// First refinement level of the prototype trees (bf16 caches): the choice of
// refinement for the root of every unit the build needs (App. A.3 "Recursive
// refinement rule": eq:app_binary_split, eq:app_extract_split,
// eq:app_split_choice; App. B.4 eq:app_tree_split_candidates), with the child
// prototypes of eq:app_rope_prototype, eq:app_value_prototype,
// eq:app_effective_multiplicity and their distortions eq:app_original_attention_stats
// .. eq:app_node_and_drop_distortion.
//
// Every unit has exactly one node to refine here, so nothing of the unit has
// to stay resident between nodes, and the workgroup is sized for two per CU
// (256 threads, under 80 KB of LDS): while one workgroup waits at a barrier or
// on memory, the other one computes.  Per unit:
//   * candidates: curvature ranks of the positions t in [0, n-2] (cut t + 1),
//     the midpoint, the extraction token (largest probe mass), all in local
//     positions; prefix children [0, x) and suffix children [x, n);
//   * child sums on the matrix cores: row c of the A operand masks the
//     tokens of child c (prefix [0, x) or suffix [x, n)); the B operand is
//     k° = RoPE^{-1}(k) (staged in fp32 one half of the dimensions at a time,
//     the pair (i, i + d/2) rotated together) or (R_t, ||k°_t||); fp32
//     operands go in three bf16 parts, so every product is exact and only the
//     fp32 accumulation rounds;
//   * child keys k~ = RoPE(mean k°, p), coherence, multiplicity, then
//     z = m_eff exp(k~ . q / sqrt(d) - m_q) for every child and probe on the
//     matrix cores (k~ split in three bf16 parts: exact products), held in
//     registers in the layout the scoring reads;
//   * distortions from the Gram matrix G = V V^T of the node (bf16 products,
//     exact; stored as 16 x 16 tiles in three bf16 parts).  For a child C and
//     probe q, ||M_q||^2, <M_q, v~_C> and ||v~_C||^2 are quadratic forms in G
//     over C's token pairs; for the nested prefix children [0, x) (suffix
//     children [x, n)) each is a sum over the child of per-token increments
//     built from Y_t = sum_{t' < t} G_tt' e_t' (t' > t), so one product
//     Y = G E^T per direction (strictly lower or upper tiles) and one masked
//     sum per child on the matrix cores replace the per-cut value sums M^T.
//     The value term ||M - z v~||^2 = ||M||^2 - 2 z <M, v~> + z^2 ||v~||^2
//     (clamped at 0) carries a rounding error of a few fp32 ulps of ||M||^2,
//     about 1e-6 of the node's attention mass in D, far below the distortions
//     compared;
//   * the fp32 scores decide (binary form wins ties, smaller cut wins ties)
//     and the root and its children are written to the node table.
#include "common.h"

namespace gkv {

constexpr int SR_T = 256;               // threads: four waves, one probe tile each
constexpr int SR_CM = CAND_MAX;         // children per direction
constexpr int SR_CC = 2 * SR_CM;        // prefix side [0, SR_CM), suffix side [SR_CM, SR_CC)

template <int D>
struct SrLds {
  static constexpr int H2 = D / 2;
  static constexpr int NTM = NMAX / 16;                   // 16-token tiles
  static constexpr int KTS = D + 4;                       // child key row stride (fp32)
  static constexpr int KOB = NMAX * (H2 + 4) * 4;         // one half of k° [NMAX][H2 + 4] fp32
  static constexpr int LDVR = D + 8;                      // staged value rows (bf16), over the k° half
  static_assert(NMAX * LDVR * 2 <= KOB, "value rows fit the k° half");
  static constexpr int KTB = SR_CC * KTS * 4;             // child k° sums -> k~
  static constexpr int GTB = 3 * 256 * 2;                 // one Gram tile: three bf16 planes of 16 x 16
  static constexpr int GB = NTM * (NTM + 1) / 2 * GTB;    // the Gram tiles (a >= b)
  // k° halves, then the Gram tiles over them and over the child keys (read
  // for the last time by the z products)
  static constexpr int oX = 0;
  static constexpr int oKt = (KOB > GB - KTB ? KOB : GB - KTB);   // [SR_CC][KTS]
  static constexpr int oCs = (oKt + KTB > GB ? oKt + KTB : GB);   // [8][SR_CC] per-child scalars
  static constexpr int oCon = oCs + 8 * SR_CC * 4;        // [SR_CC][4] per-wave D partials
  static constexpr int oPart = oCon + SR_CC * 4 * 4;      // [SR_CC][D/16] partial norms, [SR_CC][12] sums
  static constexpr int oAG = oPart + ((D / 16) + 12) * SR_CC * 4;   // [4][NMAX] rows of G against R and 1
  static constexpr int oGd = oAG + 4 * NMAX * 4;          // [NMAX] G_tt
  static constexpr int oLo = oGd + NMAX * 4;              // [Gram tiles][16] lower partial rows (R, 1)
  static constexpr int oUp = oLo + NTM * (NTM + 1) / 2 * 16 * 8;   // [Gram tiles][16] upper partials
  static constexpr int oR = oUp + NTM * (NTM + 1) / 2 * 16 * 8;    // [NMAX] R_t
  static constexpr int oA = oR + NMAX * 4;                // [NMAX] probe mass A_t
  static constexpr int oKap = oA + NMAX * 4;              // [NMAX] kappa_t
  static constexpr int oKn = oKap + NMAX * 4;             // [NMAX] ||k°_t||^2, then ||k°_t||
  static constexpr int oFlag = oKn + NMAX * 4;            // [NMAX] candidate cut flags
  static constexpr int oL = oFlag + NMAX * 4;             // lists and metadata (int)
  static constexpr int oFl = oL + 192 * 4;                // [NMAX] singleton-floor candidate flags
  static constexpr int bytes = oFl + NMAX;
};

int split_root_lds_bytes(int d) { return d == 128 ? SrLds<128>::bytes : SrLds<64>::bytes; }

// x = hi + mid + lo exactly, each a bf16, packed two per 32-bit word
__device__ __forceinline__ void sr_split3(const float* x, u32x2& hi, u32x2& mid, u32x2& lo) {
  uint32_t h[4], m[4], l[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    h[r] = __float_as_uint(x[r]) & 0xffff0000u;
    const float r1 = x[r] - __uint_as_float(h[r]);
    m[r] = __float_as_uint(r1) & 0xffff0000u;
    l[r] = __float_as_uint(r1 - __uint_as_float(m[r]));
  }
#define GKV_HI2(a, b) __builtin_amdgcn_perm((b), (a), 0x07060302u)
  hi.x = GKV_HI2(h[0], h[1]); hi.y = GKV_HI2(h[2], h[3]);
  mid.x = GKV_HI2(m[0], m[1]); mid.y = GKV_HI2(m[2], m[3]);
  lo.x = GKV_HI2(l[0], l[1]); lo.y = GKV_HI2(l[2], l[3]);
#undef GKV_HI2
}
__device__ __forceinline__ s16x4 sr_op(u32x2 v) { return __builtin_bit_cast(s16x4, v); }
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

// LV: a depth below the roots (the level list and results; mode BUILD_LEVEL or
// BUILD_LEVEL_FULL), else the roots (mode BUILD_ROOT_SPLIT or BUILD_ROOT_FULL)
template <int D, bool LV>
__global__ __launch_bounds__(SR_T, 2) void k_split_root(const Dims* __restrict__ dmp, int mode, int lvl,
                                                         const uint16_t* __restrict__ K,
                                                         const uint16_t* __restrict__ V,
                                                         const uint16_t* __restrict__ Q,
                                                         const float* __restrict__ cosT,
                                                         const float* __restrict__ sinT,
                                                         const int32_t* __restrict__ slot_starts,
                                                         const int32_t* __restrict__ n_slots,
                                                         const float* __restrict__ kappa,
                                                         const TreeView* __restrict__ tvp) {
  // the argument structures are read from device memory where used
  const Dims& dm = *dmp;
  const TreeView& tv = *tvp;
  using Lay = SrLds<D>;
  constexpr int H2 = D / 2;
  constexpr int QE = D / 4;                // dims of a probe quarter row
  constexpr int QW = QE / 2;               // 32-bit words of it
  constexpr int CT = (SR_CC + 15) / 16;    // 16-wide child tiles
  constexpr int NTM = Lay::NTM;            // 16-token tiles
  extern __shared__ __align__(16) char smem[];
  float* sKo = (float*)(smem + Lay::oX);
  uint16_t* sG = (uint16_t*)(smem + Lay::oX);
  float* sKt = (float*)(smem + Lay::oKt);
  float* sCs = (float*)(smem + Lay::oCs);
  float* sCon = (float*)(smem + Lay::oCon);
  float* sPart = (float*)(smem + Lay::oPart);
  float* sR = (float*)(smem + Lay::oR);
  float* sA = (float*)(smem + Lay::oA);
  float* sKap = (float*)(smem + Lay::oKap);
  float* sKn = (float*)(smem + Lay::oKn);
  float* sAG = (float*)(smem + Lay::oAG);
  float* sGd = (float*)(smem + Lay::oGd);
  float2* sLo = (float2*)(smem + Lay::oLo);
  float2* sUp = (float2*)(smem + Lay::oUp);
  int* sFlag = (int*)(smem + Lay::oFlag);
  uint8_t* sFl = (uint8_t*)(smem + Lay::oFl);
  int* XL = (int*)(smem + Lay::oL);        // [0, 32)   prefix cuts (child [0, x))
  int* XR = XL + 32;                       // [32, 64)  suffix cuts (child [x, n))
  int* XB = XL + 64;                       // [64, 96)  binary cuts
  int* posL = XL + 96;                     // index of XB[k] in XL
  int* posR = XL + 128;                    // index of XB[k] in XR
  int* meta = XL + 160;                    // nl, nr, nb, p, kmin, kmax, index of p in XL, of p+1 in XR,
                                           // forced extraction (singleton floor), work item
  auto crow = [&](int r) { return sCs + r * SR_CC; };

  const int tid0 = threadIdx.x;
  const int J = *n_slots;
  // roots: the build's work list; a level (depth lvl >= 1): that depth's list,
  // its length in lv_ctr[lvl & 1], the next item in lv_ctr[2]
  constexpr bool level = LV;
  const int32_t* items = level ? tv.lv_items : tv.work;
  int32_t* next_ctr = level ? tv.lv_ctr + 2 : tv.wctr + 1;
  const int nwork = level ? (int)min((int64_t)tv.lv_ctr[lvl & 1], tv.lv_cap) : tv.wctr[0];
  if (level && blockIdx.x == 0 && tid0 == 0) {
    // the counters the level pass after this kernel accumulates into: the next
    // depth's items and units
    tv.lv_ctr[(lvl + 1) & 1] = 0;
    tv.lv_ctr[4 + ((lvl + 1) & 1)] = 0;
  }
  const float scale = 1.0f / sqrtf((float)D);
  const float LOG2E = 1.44269504088896341f;

  if (tid0 == 0) meta[9] = atomicAdd(next_ctr, 1);
  for (;;) {
    // per-lane indices are formed inside the loop (values derived from them are
    // not held across items, which would not fit the register budget)
    int tid = tid0;
    asm volatile("" : "+v"(tid));
    const int wave = uni(tid >> 6), lane = tid & 63, i16 = lane & 15, g4 = lane >> 4;
    const int pt = wave;                     // probe tile of this wave
    const int q = 16 * pt + i16;             // the lane's probe (scoring layout)
    const bool pok = q < dm.W;
    sync_after_lds_stores();                 // meta[9] was stored at the end of the last pass
    const int wi = uni(meta[9]);
    __syncthreads();
    if (wi >= nwork) break;
    // the next item, in flight while this one is processed (stored before the
    // barrier at the top of the next pass)
    int wnext = 0;
    if (tid == 0) wnext = atomicAdd(next_ctr, 1);
    auto publish_next = [&]() { if (tid == 0) meta[9] = wnext; };
    do {
    // the work item: unit, the node's start, length (and BFS index), D and R, w
    // and the key of the op that creates it (one load)
    const int4 d0 = *(const int4*)(items + 8 * (int64_t)wi);
    const int4 d1 = *(const int4*)(items + 8 * (int64_t)wi + 4);
    const int64_t unit = uni(d0.x);
    const int lg = (int)(unit / dm.J_cap), j = (int)(unit % dm.J_cap);
    const int l = lg / dm.G, g = lg % dm.G;
    const int a0 = uni(d0.y);
    const int n = uni(d0.z) & 0xffff;
    const float Dv = __int_as_float(uni(d0.w));
    const float Rroot = __int_as_float(uni(d1.x));
    const float w = __int_as_float(uni(d1.y));
    const uint64_t Eadd = mode == BUILD_ROOT_FULL ? 0ull
                                                  : ((uint64_t)(uint32_t)uni(d1.w) << 32) | (uint32_t)uni(d1.z);
    if (n < 2 || n > NMAX || j >= J) break;
    const int64_t base = (int64_t)lg * 2 * dm.N_c + 2 * (int64_t)a0;
    const uint32_t ord = (uint32_t)lg * (uint32_t)J + (uint32_t)j;
    const uint16_t* Kp = K + ((int64_t)lg * dm.T + a0) * D;
    const uint16_t* Vp = V + ((int64_t)lg * dm.T + a0) * D;
    const float* tokR = tv.tok_R + (int64_t)lg * dm.N_c + a0;
    // ---- writes the root and its children (local positions), or a level's
    // result: kind | nkid << 8 | cut << 16, U, then per child (start | length << 16),
    // D, R (node-local positions; the level pass numbers and places them) ----
    auto write_tree = [&](int kind, int cut, int nkid, const int* ka, const int* kn, const float* kD,
                          const float* kR) {
      if constexpr (level) {
        float sd = 0.f;
        for (int k = 0; k < nkid; ++k) sd += kD[k];
        const float Us = utility(split_gain(w, Rroot, Dv, sd), nkid - 1);
        int4* r = (int4*)(tv.lv_res + 12 * (int64_t)wi);
        const int k2 = nkid > 2 ? ka[2] | (kn[2] << 16) : 0;
        r[0] = make_int4(kind | (nkid << 8) | (cut << 16), __float_as_int(Us), ka[0] | (kn[0] << 16), ka[1] | (kn[1] << 16));
        r[1] = make_int4(k2, __float_as_int(kD[0]), __float_as_int(kD[1]), nkid > 2 ? __float_as_int(kD[2]) : 0);
        r[2] = make_int4(__float_as_int(kR[0]), __float_as_int(kR[1]), nkid > 2 ? __float_as_int(kR[2]) : 0, 0);
        return;
      }
      tv.node_child[base] = 1;
      tv.node_nch[base] = (uint8_t)nkid;
      tv.node_kind[base] = (uint8_t)kind;
      tv.node_cut[base] = a0 + cut;
      float sd = 0.f;
      for (int k = 0; k < nkid; ++k) {
        const int64_t s = base + 1 + k;
        tv.node_a[s] = a0 + ka[k];
        tv.node_n[s] = kn[k];
        tv.node_child[s] = -1;
        tv.node_parent[s] = 0;
        tv.node_nch[s] = 0;
        tv.node_kind[s] = 0;
        tv.node_cut[s] = -1;
        tv.node_D[s] = kD[k];
        tv.node_R[s] = kR[k];
        tv.sp_U[s] = 0.f;
        tv.sp_E[s] = 0;
        tv.sp_cost[s] = 0;
        tv.sp_exec[s] = 0;
        sd += kD[k];
      }
      if (mode != BUILD_ROOT_FULL) {        // the root's Split key, known now
        const float Us = utility(split_gain(w, Rroot, Dv, sd), nkid - 1);
        const uint64_t k = op_key(Us, ord * 256u + 1u);
        tv.sp_U[base] = Us;
        tv.sp_E[base] = k < Eadd ? k : Eadd;
        tv.sp_cost[base] = (uint8_t)(nkid - 1);
        tv.sp_exec[base] = 0;
      }
      tv.unit_nn[unit] = 1 + nkid;
    };
    if (n == 2) {                            // one cut, two singletons
      if (tid == 0) {
        const int ka[2] = {0, 1}, kn[2] = {1, 1};
        const float kD[2] = {0.f, 0.f}, kR[2] = {tokR[0], tokR[1]};
        write_tree(1, 1, 2, ka, kn, kD, kR);
      }
      break;
    }

    // ---- staging: token values, probe masses, curvature, probe rows ----
    constexpr int CH = H2 / 8;
    constexpr int IPT = (NMAX * CH + SR_T - 1) / SR_T;   // k° items (token, 8-dim chunk) per thread
    float rv = 0.f, av = 0.f, kv = 0.f;
    uint8_t fl = 0;
    if (tid < n) {
      rv = tokR[tid];
      av = tv.tok_A[(int64_t)lg * dm.N_c + a0 + tid];
      kv = kappa[a0 + tid];
      if (tv.fl_flag) fl = tv.fl_flag[(int64_t)lg * dm.N_c + a0 + tid];
    }
    // probe shift and normaliser of the lane's probe (probe q: window query q of
    // head q mod |H(g)|); its row is loaded with the child keys
    float mq2 = 0.f, izc = 1.f;
    if (pok) {
      mq2 = tv.probe_m[(int64_t)lg * dm.W + q] * LOG2E;
      izc = 1.0f / tv.probe_ZC[(int64_t)lg * dm.W + q];
    }
    if (tid < n) {
      sR[tid] = rv;
      sA[tid] = av;
      sKap[tid] = kv;
      sFl[tid] = fl;
    }
    for (int t = tid; t < NMAX; t += SR_T) sFlag[t] = 0;
    __syncthreads();
    // curvature position t proposes the cut t + 1; top k_curv by kappa over
    // [0, n-2], ties to the smaller t; midpoint floor(n/2)
    if (dm.k_curv > 0 && tid < n - 1) {
      const float kt = sKap[tid];
      int rank = 0;
      const int hi = n - 2;
      for (int t4 = 0; t4 <= hi; t4 += 8) {
        const float4 k4 = *(const float4*)(sKap + t4);
        const float4 k5 = *(const float4*)(sKap + t4 + 4);
        const float kk[8] = {k4.x, k4.y, k4.z, k4.w, k5.x, k5.y, k5.z, k5.w};
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
          const int t2 = t4 + jj;
          rank += (int)((t2 <= hi) & ((kk[jj] > kt) | ((kk[jj] == kt) & (t2 < tid))));
        }
      }
      if (rank < dm.k_curv) sFlag[tid + 1] = 1;
    }
    if (tid == SR_T - 1) sFlag[n / 2] = 1;
    if (wave == 3) {                         // curvature range and extraction token
      float kmn = INFINITY, kmx = -INFINITY, best = -INFINITY, bestf = -INFINITY;
      int bi = 0x7fffffff, bf = 0x7fffffff;
      for (int t = lane; t < n; t += 64) {
        const float k = sKap[t];
        kmn = fminf(kmn, k);
        kmx = fmaxf(kmx, k);
        const float am = sA[t];
        if (am > best || (am == best && t < bi)) { best = am; bi = t; }
        // singleton floor: the candidate of largest token value (App. A.3 split choice)
        if (sFl[t] && (sR[t] > bestf || (sR[t] == bestf && t < bf))) { bestf = sR[t]; bf = t; }
      }
      wave_minmax(kmn, kmx);
      wave_argmax(best, bi);
      wave_argmax(bestf, bf);
      if (lane == 0) {
        // a node of three or more tokens holding a floor candidate is extracted
        // there, with no choice
        const bool forced = bf != 0x7fffffff;
        meta[3] = forced ? bf : bi;
        meta[4] = __float_as_int(kmn);
        meta[5] = __float_as_int(kmx);
        meta[8] = forced ? 1 : 0;
      }
    }
    __syncthreads();
    // binary cuts XB ascending (by ballot over the flags), then XL = XB + {p}
    // (p > 0) and XR = XB + {p+1} (p+1 < n)
    if (wave == 0) {
      const bool forced = meta[8] != 0;        // extraction only: no binary cut
      const bool f0 = !forced && lane >= 1 && lane < n && sFlag[lane];
      const bool f1 = !forced && 64 + lane < n && sFlag[64 + lane];
      const uint64_t m0 = __ballot(f0), m1 = __ballot(f1);
      const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
      const int c0 = __popcll(m0);
      if (f0) XB[__popcll(m0 & below)] = lane;
      if (f1) XB[c0 + __popcll(m1 & below)] = 64 + lane;
      if (lane == 0) meta[2] = c0 + __popcll(m1);
    }
    __syncthreads();
    if (wave == 0) {
      const int nb = meta[2], p = meta[3];
      const bool on = lane < nb;
      const int xb = on ? XB[lane] : 0x7fffffff;
      const bool useP = p > 0, useQ = p + 1 < n;
      const uint64_t lessP = __ballot(on && xb < p), eqP = __ballot(on && xb == p);
      const uint64_t lessQ = __ballot(on && xb < p + 1), eqQ = __ballot(on && xb == p + 1);
      const bool insL = useP && eqP == 0ull, insR = useQ && eqQ == 0ull;
      if (on) {
        const int pl = lane + ((insL && xb > p) ? 1 : 0);
        const int pr = lane + ((insR && xb > p + 1) ? 1 : 0);
        XL[pl] = xb; posL[lane] = pl;
        XR[pr] = xb; posR[lane] = pr;
      }
      if (lane == 0) {
        const int cp = __popcll(lessP), cq = __popcll(lessQ);
        if (insL) XL[cp] = p;
        if (insR) XR[cq] = p + 1;
        meta[0] = nb + (insL ? 1 : 0);
        meta[1] = nb + (insR ? 1 : 0);
        meta[6] = useP ? cp : -1;
        meta[7] = useQ ? cq : -1;
      }
    }
    __syncthreads();
    const int nl = uni(meta[0]), nr = uni(meta[1]), nb = uni(meta[2]), p = uni(meta[3]);

    // ---- children's sums on the matrix cores ----
    // A operand rows = children (row gc: prefix child gc < SR_CM covers [0, XL[gc]),
    // suffix child gc - SR_CM covers [XR[gc - SR_CM], n)), as a 0/1 mask or the
    // masked token values; B operand = the tokens' k° or v (k° and R split in
    // three bf16 parts: exact products, fp32 accumulation).  Lane (i16, g4)
    // feeds row 16 ct + i16 and tokens 16 s + 4 g4 + r.
    // bf16 1.0 (as 0xffff masks) per token t0 .. t0 + 3 inside child row 16 ct + i16
    auto row_bounds = [&](int ct, int& lo, int& hi) {
      const int gc = 16 * ct + i16;
      lo = 0;
      hi = 0;
      if (gc < SR_CM) {
        if (gc < nl) hi = XL[gc];
      } else if (gc < SR_CC && gc - SR_CM < nr) {
        lo = XR[gc - SR_CM];
        hi = n;
      }
    };
    auto mask16 = [&](int lo, int hi, int t0) {
      uint32_t m[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) m[r] = (t0 + r >= lo && t0 + r < hi) ? 0xffffu : 0u;
      u32x2 v;
      v.x = m[0] | (m[1] << 16);
      v.y = m[2] | (m[3] << 16);
      return v;
    };
    const u32x2 one2 = {0x3F803F80u, 0x3F803F80u};   // bf16 1.0 in every half
    const int nks = (n + 15) >> 4;           // 16-token k steps
    constexpr int NP = D / 16;               // 16-dim partials per child
    float* sPss = sPart;                     // [SR_CC][NP] ||mean k°||^2 partials
    float* sTmp = sPart + SR_CC * NP;        // [SR_CC][12] sums in three parts each
    // lengths of the children (0: no such child)
    if (tid < SR_CC) {
      int nch = 0;
      if (tid < SR_CM) { if (tid < nl) nch = XL[tid]; }
      else if (tid - SR_CM < nr) nch = n - XR[tid - SR_CM];
      crow(0)[tid] = (float)nch;
    }

    // ---- key sums: k° staged one half of the dims at a time ----
    constexpr int KSTR = H2 + 4;             // k° row stride (fp32): conflict-free column reads
    constexpr int HT = H2 / 16;              // 16-dim tiles per half
    for (int hf = 0; hf < 2; ++hf) {
      // k° of the half (item (token, 8-dim chunk): the pair (i, i + H2) is
      // rotated together), turned back to the node's start a0: the table row of
      // the offset t (R_{p~} R_{a0 + t}^{-1} = R_{p~ - a0} R_t^{-1}; rows below
      // NMAX stay cached); every load of the half in flight first
      uint32_t kw1[IPT][4], kw2[IPT][4];
      float cs[IPT][8], sn[IPT][8];
#pragma unroll
      for (int it = 0; it < IPT; ++it) {
        const int e = tid + SR_T * it;
        const int ee = e < n * CH ? e : 0;
        const int t = ee / CH, c = 8 * (ee % CH);
        const int64_t ta = t;
        const uint4 u1 = *(const uint4*)(Kp + (int64_t)t * D + c);
        const uint4 u2 = *(const uint4*)(Kp + (int64_t)t * D + c + H2);
        const float4 c0 = *(const float4*)(cosT + ta * H2 + c), c1 = *(const float4*)(cosT + ta * H2 + c + 4);
        const float4 s0 = *(const float4*)(sinT + ta * H2 + c), s1 = *(const float4*)(sinT + ta * H2 + c + 4);
        kw1[it][0] = u1.x; kw1[it][1] = u1.y; kw1[it][2] = u1.z; kw1[it][3] = u1.w;
        kw2[it][0] = u2.x; kw2[it][1] = u2.y; kw2[it][2] = u2.z; kw2[it][3] = u2.w;
        cs[it][0] = c0.x; cs[it][1] = c0.y; cs[it][2] = c0.z; cs[it][3] = c0.w;
        cs[it][4] = c1.x; cs[it][5] = c1.y; cs[it][6] = c1.z; cs[it][7] = c1.w;
        sn[it][0] = s0.x; sn[it][1] = s0.y; sn[it][2] = s0.z; sn[it][3] = s0.w;
        sn[it][4] = s1.x; sn[it][5] = s1.y; sn[it][6] = s1.z; sn[it][7] = s1.w;
      }
#pragma unroll
      for (int it = 0; it < IPT; ++it) {
        const int e = tid + SR_T * it;
        if (e >= n * CH) break;
        const int t = e / CH, c = 8 * (e % CH);
        float o[8];
        float ss = 0.f;
#pragma unroll
        for (int h = 0; h < 8; ++h) {
          const float k1 = (h & 1) ? __uint_as_float(kw1[it][h >> 1] & 0xffff0000u) : __uint_as_float(kw1[it][h >> 1] << 16);
          const float k2 = (h & 1) ? __uint_as_float(kw2[it][h >> 1] & 0xffff0000u) : __uint_as_float(kw2[it][h >> 1] << 16);
          o[h] = hf == 0 ? k1 * cs[it][h] + k2 * sn[it][h] : k2 * cs[it][h] - k1 * sn[it][h];
          ss += o[h] * o[h];
        }
        float4* d1 = (float4*)(sKo + t * KSTR + c);
        d1[0] = make_float4(o[0], o[1], o[2], o[3]);
        d1[1] = make_float4(o[4], o[5], o[6], o[7]);
        // ||k°_t||^2: the CH items of token t sit in CH consecutive lanes
#pragma unroll
        for (int ob = 1; ob < CH; ob <<= 1) ss += __shfl_xor(ss, ob, 64);
        if (e % CH == 0) sKn[t] = hf == 0 ? ss : sKn[t] + ss;
      }
      __syncthreads();
      // wave = 16-dim tile of the half: every child's sum, and the partial of
      // ||mean k°||^2 over the tile's dims
      for (int tile = wave; tile < HT; tile += SR_T / 64) {
        int clo[CT], chi[CT];
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) row_bounds(ct, clo[ct], chi[ct]);
        f32x4 acc[CT];
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
        // 16-token steps in pairs on the 16x16x32 instruction (the lane's four
        // tokens of step s, then of step s + 1, on both sides)
        auto cat2 = [](u32x2 a, u32x2 b) { return pk8(make_uint4(a.x, a.y, b.x, b.y)); };
        for (int s = 0; s < nks; s += 2) {
          u32x2 kh[2], km[2], kl[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int t0 = 16 * (s + h) + 4 * g4;
            float x[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) x[r] = t0 + r < n ? sKo[(t0 + r) * KSTR + 16 * tile + i16] : 0.f;
            sr_split3(x, kh[h], km[h], kl[h]);
          }
          const int ta = 16 * s + 4 * g4, tb = ta + 16;
          const s16x8 bl = cat2(kl[0], kl[1]), bm = cat2(km[0], km[1]), bh = cat2(kh[0], kh[1]);
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) {
            const s16x8 mk = cat2(one2 & mask16(clo[ct], chi[ct], ta), one2 & mask16(clo[ct], chi[ct], tb));
            acc[ct] = mfma_bf16_16x16x32(mk, bl, acc[ct]);
            acc[ct] = mfma_bf16_16x16x32(mk, bm, acc[ct]);
            acc[ct] = mfma_bf16_16x16x32(mk, bh, acc[ct]);
          }
        }
        // lane (dim 16 tile + i16, g4) holds children 16 ct + 4 g4 + r
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int gr = 16 * ct + 4 * g4 + r;
            const int grr = gr < SR_CC ? gr : 0;
            const float nch = crow(0)[grr];
            const float inv = nch > 0.f ? 1.0f / nch : 0.f;
            const float m = acc[ct][r] * inv;
            const float ps = row_sum16(m * m);
            if (gr < SR_CC) {
              sKt[gr * Lay::KTS + hf * H2 + 16 * tile + i16] = acc[ct][r];
              if (i16 == 0) sPss[gr * NP + hf * HT + tile] = ps;
            }
          }
      }
      __syncthreads();
    }

    if (tid < n) sKn[tid] = sqrtf(sKn[tid]);
    // the node's values, row-major bf16 into the k° half (free from here on):
    // every load in flight now, stored after the child keys; rows past the
    // node up to the last 16-token tile are zero
    const int nt = (n + 15) >> 4;            // 16-token tiles
    constexpr int VCH = D / 8;               // 16-byte chunks of a row
    constexpr int VIT = NMAX * VCH / SR_T;   // (row, chunk) items per thread
    uint4 vst[VIT];
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
      const int e = tid + SR_T * it;
      const int t = e / VCH, c = e % VCH;
      vst[it] = make_uint4(0u, 0u, 0u, 0u);
      if (t < n) vst[it] = *(const uint4*)(Vp + (int64_t)t * D + 8 * c);
    }
    __syncthreads();
    // sum R and sum ||k°|| of every child: wave = child tile; B columns 0-2 hold
    // R in three parts, columns 3-5 ||k°|| in three parts
    if (wave < CT) {
      const int ct = wave;
      int clo, chi;
      row_bounds(ct, clo, chi);
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
      const int part = i16 % 3;
      const float* src = i16 < 3 ? sR : sKn;
      for (int s = 0; s < nks; ++s) {
        const int t0 = 16 * s + 4 * g4;
        float x[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) x[r] = (i16 < 6 && t0 + r < n) ? src[t0 + r] : 0.f;
        u32x2 xh, xm, xl;
        sr_split3(x, xh, xm, xl);
        const u32x2 b = part == 0 ? xh : (part == 1 ? xm : xl);
        acc = mfma_bf16_16x16x16(sr_op(one2 & mask16(clo, chi, t0)), sr_op(b), acc);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int gr = 16 * ct + 4 * g4 + r;
        if (gr < SR_CC && i16 < 6) sTmp[gr * 12 + i16] = acc[r];
      }
    }
    __syncthreads();
    if (tid < SR_CC) {
      const float* x = sTmp + tid * 12;
      const float nch = crow(0)[tid];
      crow(1)[tid] = x[2] + x[1] + x[0];
      crow(2)[tid] = nch > 0.f ? (x[5] + x[4] + x[3]) / nch : 0.f;
    }
    __syncthreads();
    // ---- child keys: coherence, multiplicity (eq:app_effective_multiplicity),
    // k~ = RoPE(mean k°, p) (eq:app_rope_prototype) ----
    // the probe quarter rows of the wave's tile, in flight meanwhile
    uint32_t qreg[QW];
    {
      const int uq = pok ? q : 0;
      const uint16_t* Qp = Q + ((int64_t)l * dm.H + (int64_t)g * dm.hpg) * dm.W * D;
      const uint4* q4 = (const uint4*)(Qp + ((int64_t)(uq % dm.hpg) * dm.W + uq) * D + QE * g4);
#pragma unroll
      for (int h = 0; h < QW / 4; ++h) {
        const uint4 v = q4[h];
        qreg[4 * h] = v.x; qreg[4 * h + 1] = v.y; qreg[4 * h + 2] = v.z; qreg[4 * h + 3] = v.w;
      }
    }
    if (tid < SR_CC) {
      const float nch = crow(0)[tid];
      if (nch >= 2.f) {
        float ss = 0.f;
#pragma unroll
        for (int k = 0; k < NP; ++k) ss += sPss[tid * NP + k];
        const float coh = sqrtf(ss) / (crow(2)[tid] + dm.eps);
        crow(3)[tid] = fminf(fmaxf(nch * coh * coh, 1.0f), nch);
      }
    }
    {
      constexpr int RPT = (SR_CC * H2 + SR_T - 1) / SR_T;   // (child, pair) items per thread
      float ccv[RPT], snv[RPT];
#pragma unroll
      for (int m = 0; m < RPT; ++m) {         // the rotation rows, every load in flight together
        const int e = tid + SR_T * m;
        const int gc = e / H2, i = e % H2;
        int64_t pp = 0;                      // the child's representative position less a0
        if (e < SR_CC * H2) {
          const int nch = (int)crow(0)[gc];
          if (nch >= 2) {
            const int x0 = gc < SR_CM ? 0 : XR[gc - SR_CM];
            pp = round_half_even_mid(a0 + x0, a0 + x0 + nch) - a0;
          }
        }
        ccv[m] = cosT[pp * H2 + i];
        snv[m] = sinT[pp * H2 + i];
      }
#pragma unroll
      for (int m = 0; m < RPT; ++m) {
        const int e = tid + SR_T * m;
        if (e >= SR_CC * H2) break;
        const int gc = e / H2, i = e % H2;
        const float nch = crow(0)[gc];
        if (nch < 2.f) continue;
        const float inv = 1.0f / nch;
        float* kt = sKt + gc * Lay::KTS;
        const float m1 = kt[i] * inv, m2 = kt[i + H2] * inv;
        kt[i] = m1 * ccv[m] - m2 * snv[m];
        kt[i + H2] = m2 * ccv[m] + m1 * snv[m];
      }
    }
    uint16_t* sVr = (uint16_t*)(smem + Lay::oX);
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
      const int e = tid + SR_T * it;
      const int t = e / VCH, c = e % VCH;
      if (t < 16 * nt) *(uint4*)(sVr + t * Lay::LDVR + 8 * c) = vst[it];
    }
    __syncthreads();

    // the keys of the first 16-token tile, in flight during the z products
    auto kload = [&](int j, uint32_t* dst) {
      int tr = 16 * j + i16;
      tr = tr < n ? tr : n - 1;
      const uint4* k4 = (const uint4*)(Kp + (int64_t)tr * D + QE * g4);
#pragma unroll
      for (int h = 0; h < QW / 4; ++h) {
        const uint4 v = k4[h];
        dst[4 * h] = v.x; dst[4 * h + 1] = v.y; dst[4 * h + 2] = v.z; dst[4 * h + 3] = v.w;
      }
    };
    const int np = nt * (nt + 1) / 2;        // Gram tiles
    auto tile_ab = [&](int k, int& a, int& b) {
      a = 0;
      while ((a + 1) * (a + 2) / 2 <= k) ++a;
      b = k - a * (a + 1) / 2;
    };
    uint32_t kcur[QW];
    kload(0, kcur);

    // ---- z_{q,c} = m_eff exp(k~_c . q / sqrt(d) - m_q): child rows x probe columns
    // on the matrix cores; lane (i16 = probe, g4) holds children 16 ct + 4 g4 + r ----
    float zreg[CT][4];
    {
      const float sc2 = scale * LOG2E;
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        const int gc = 16 * ct + i16;        // the child row this lane feeds
        const int gcc = gc < SR_CC ? gc : 0;
        const bool live = gc < SR_CC && ((gc < SR_CM && gc < nl) || (gc >= SR_CM && gc - SR_CM < nr));
        const bool cok = live && crow(0)[gcc] >= 2.f;
        const float* kt = sKt + gcc * Lay::KTS + QE * g4;
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < QE / 4; ++s) {
          float x[4];
          const float4 v = *(const float4*)(kt + 4 * s);
          x[0] = cok ? v.x : 0.f; x[1] = cok ? v.y : 0.f; x[2] = cok ? v.z : 0.f; x[3] = cok ? v.w : 0.f;
          u32x2 h, m, lo;
          sr_split3(x, h, m, lo);
          const s16x4 qb = pk4(qreg[2 * s], qreg[2 * s + 1]);
          acc = mfma_bf16_16x16x16(sr_op(lo), qb, acc);
          acc = mfma_bf16_16x16x16(sr_op(m), qb, acc);
          acc = mfma_bf16_16x16x16(sr_op(h), qb, acc);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int gr = 16 * ct + 4 * g4 + r;
          const float me = gr < SR_CC ? crow(3)[gr] : 1.f;
          zreg[ct][r] = __builtin_amdgcn_exp2f(acc[r] * sc2 - mq2) * me;
        }
      }
    }
    // ---- probe exponentials e_{q,t} = exp(q . k_t / sqrt(d) - m_q) of every token
    // (transposed logits on the matrix cores): lane (i16 = probe, g4) holds tokens
    // 16 j + 4 g4 + r of tile j, in fp32 and in three bf16 parts ----
    const bool probes = 16 * pt < dm.W;
    u32x2 eh[NTM], em[NTM], el[NTM];
    if (probes) {
      const float sc2 = scale * LOG2E;
#pragma unroll
      for (int j = 0; j < NTM; ++j) {
        if (j < nt) {
          uint32_t knext[QW];
          if (j + 1 < nt) kload(j + 1, knext);
          f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int s = 0; s < QE / 8; ++s)
            acc = mfma_bf16_16x16x32(pk8(make_uint4(kcur[4 * s], kcur[4 * s + 1], kcur[4 * s + 2], kcur[4 * s + 3])),
                                     pk8(make_uint4(qreg[4 * s], qreg[4 * s + 1], qreg[4 * s + 2], qreg[4 * s + 3])),
                                     acc);
          float ev[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int t = 16 * j + 4 * g4 + r;
            // exp2(-inf) = 0 for the masked ones: no branch around the exponential
            ev[r] = __builtin_amdgcn_exp2f((pok && t < n) ? acc[r] * sc2 - mq2 : -INFINITY);
          }
          sr_split3(ev, eh[j], em[j], el[j]);
          if (j + 1 < nt) {
#pragma unroll
            for (int h = 0; h < QW; ++h) kcur[h] = knext[h];
          }
        } else {
          // defined on every path: an undefined value would be carried from
          // item to item, and kept in registers across the whole loop
          eh[j] = u32x2{0u, 0u};
          em[j] = eh[j];
          el[j] = eh[j];
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < NTM; ++j) {
        eh[j] = u32x2{0u, 0u};
        em[j] = eh[j];
        el[j] = eh[j];
      }
    }
    // ---- Gram matrix of the node's values, G = V V^T (the value terms of D_q,
    // eq:app_node_and_drop_distortion, are quadratic forms in it), in 16 x 16
    // tiles a >= b, from the staged value rows; wave w takes the tiles
    // w, w + 4, ... and holds them in registers until the planes can be
    // stored.  Tile a (a + 1) / 2 + b holds G[16 a + i][16 b + j] at lane
    // i + 16 (j / 4), element j % 4 (the A-operand layout of G[a, b], and read
    // across, of G[b, a]), as three bf16 planes with G = hi + mid + lo exactly;
    // bf16 products are exact, so G carries only the fp32 accumulation.  With
    // each tile, the partial rows of G against R and 1 over t' < t: for the
    // rows t of tile a, sum over the columns t' of tile b (lower), and for the
    // columns t' of tile b, sum over the rows t of tile a (upper); tokens past
    // the node count as zero. ----
    constexpr int GTM = (NTM * (NTM + 1) / 2 + SR_T / 64 - 1) / (SR_T / 64);   // tiles per wave
    float gt[GTM][4];
#pragma unroll
    for (int m = 0; m < GTM; ++m) {
      const int k = wave + (SR_T / 64) * m;
      if (k < np) {
        int a, b;
        tile_ab(k, a, b);
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s2 = 0; s2 < D / 32; ++s2) {
          const uint4 xb = *(const uint4*)(sVr + (16 * b + i16) * Lay::LDVR + 32 * s2 + 8 * g4);
          const uint4 xa = *(const uint4*)(sVr + (16 * a + i16) * Lay::LDVR + 32 * s2 + 8 * g4);
          acc = mfma_bf16_16x16x32(pk8(xb), pk8(xa), acc);
        }
        // C[i][j] = v_{16b+i} . v_{16a+j}: lane (i16, g4) holds G[16a + i16][16b + 4 g4 + r]
        const float x[4] = {acc[0], acc[1], acc[2], acc[3]};
        if (a == b && g4 == (i16 >> 2)) {
          const int rr = i16 & 3;
          sGd[16 * a + i16] = rr == 0 ? x[0] : (rr == 1 ? x[1] : (rr == 2 ? x[2] : x[3]));
        }
        const int tr = 16 * a + i16, tc0 = 16 * b + 4 * g4;
        const float Rrow = tr < n ? sR[tr] : 0.f;
        float la = 0.f, lg = 0.f, ua[4], ug[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool keep = tc0 + r < tr && tr < n;       // t' < t < n
          const float gv = keep ? x[r] : 0.f;
          const float Rc = keep ? sR[tc0 + r] : 0.f;
          la = fmaf(gv, Rc, la);
          lg += gv;
          ua[r] = gv * Rrow;
          ug[r] = gv;
        }
        la = col_sum4(la);
        lg = col_sum4(lg);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          ua[r] = row_sum16(ua[r]);
          ug[r] = row_sum16(ug[r]);
        }
        if (g4 == 0) sLo[16 * k + i16] = make_float2(la, lg);
        if (i16 == 0) {
#pragma unroll
          for (int r = 0; r < 4; ++r) sUp[16 * k + 4 * g4 + r] = make_float2(ua[r], ug[r]);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) gt[m][r] = x[r];
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) gt[m][r] = 0.f;   // defined on every path
      }
    }
    __syncthreads();                         // child keys and value rows are read: the Gram planes go over them
#pragma unroll
    for (int m = 0; m < GTM; ++m) {
      const int k = wave + (SR_T / 64) * m;
      if (k < np) {
        u32x2 h, mi, lo;
        sr_split3(gt[m], h, mi, lo);
        u32x2* dst = (u32x2*)(sG + (size_t)k * 768);
        dst[lane] = h;
        dst[64 + lane] = mi;
        dst[128 + lane] = lo;
      }
    }
    // A operand of G[i, j] (rows: tokens of tile i, k: tokens of tile j)
    auto gread = [&](int i, int j, u32x2& h, u32x2& m, u32x2& lo) {
      if (j <= i) {
        const u32x2* src = (const u32x2*)(sG + (size_t)(i * (i + 1) / 2 + j) * 768);
        h = src[lane];
        m = src[64 + lane];
        lo = src[128 + lane];
      } else {
        // G[i, j] = G[j, i]^T: element (i16, 4 g4 + r) is element (4 g4 + r, i16) of tile (j, i)
        const uint16_t* src = sG + (size_t)(j * (j + 1) / 2 + i) * 768 + 16 * g4 + 64 * (i16 >> 2) + (i16 & 3);
        u32x2 v[3];
#pragma unroll
        for (int p3 = 0; p3 < 3; ++p3) {
          const uint16_t* pp = src + 256 * p3;
          v[p3].x = (uint32_t)pp[0] | ((uint32_t)pp[4] << 16);
          v[p3].y = (uint32_t)pp[8] | ((uint32_t)pp[12] << 16);
        }
        h = v[0];
        m = v[1];
        lo = v[2];
      }
    };
    // strictly lower (k < row) and strictly upper (k > row) parts of a diagonal tile
    u32x2 mlo, mup;
    {
      uint32_t a4[4], b4[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        a4[r] = 4 * g4 + r < i16 ? 0xffffu : 0u;
        b4[r] = 4 * g4 + r > i16 ? 0xffffu : 0u;
      }
      mlo.x = a4[0] | (a4[1] << 16); mlo.y = a4[2] | (a4[3] << 16);
      mup.x = b4[0] | (b4[1] << 16); mup.y = b4[2] | (b4[3] << 16);
    }
    __syncthreads();
    // ---- per token, a_t = sum G_tt' R_t' and g_t = sum G_tt' over t' < t (wave 0)
    // or t' > t (wave 1), summed from the partials in a fixed order; then
    // ||v~||^2 of every child (eq:app_value_prototype): with w_t = R_t + beta,
    // ||sum w_t v_t||^2 = RR + 2 beta RG + beta^2 GG with RR = sum R_t R_t' G_tt',
    // RG = sum R_t G_tt', GG = sum G_tt' over the child's token pairs, each the
    // sum over the child of a per-token increment (prefix children: lower rows
    // and a prefix scan, wave 0; suffix children: upper rows and a suffix scan,
    // wave 1); two tokens per lane. ----
    if (wave < 2) {
      const int dir = wave;
      float x0[3], x1[3];
#pragma unroll
      for (int e2 = 0; e2 < 2; ++e2) {
        const int t = 2 * lane + e2;
        const int a = t >> 4, i = t & 15;
        float av = 0.f, gv = 0.f;
        if (a < nt) {
          if (dir == 0) {
            for (int b = 0; b <= a; ++b) {
              const float2 p2 = sLo[16 * (a * (a + 1) / 2 + b) + i];
              av += p2.x;
              gv += p2.y;
            }
          } else {
            for (int a2 = a; a2 < nt; ++a2) {
              const float2 p2 = sUp[16 * (a2 * (a2 + 1) / 2 + a) + i];
              av += p2.x;
              gv += p2.y;
            }
          }
          sAG[2 * dir * NMAX + t] = av;
          sAG[(2 * dir + 1) * NMAX + t] = gv;
        }
        float q0 = 0.f, q1 = 0.f, q2 = 0.f;
        if (t < n) {
          const float R = sR[t], gd = sGd[t];
          q0 = R * (2.f * av + gd * R);
          q1 = (R * gv + av) + R * gd;
          q2 = 2.f * gv + gd;
        }
        float* xs = e2 ? x1 : x0;
        xs[0] = q0; xs[1] = q1; xs[2] = q2;
      }
      // inclusive prefix sums over t (wave 0) or suffix sums (wave 1) at both tokens of the lane
      float s0[3], s1[3];
#pragma unroll
      for (int qq = 0; qq < 3; ++qq) {
        const float tot = x0[qq] + x1[qq];
        float sc = tot;                      // scan of the lane totals, lanes before (after) this one
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const float y = dir == 0 ? __shfl_up(sc, off, 64) : __shfl_down(sc, off, 64);
          if (dir == 0 ? lane >= off : lane + off < 64) sc += y;
        }
        const float ex0 = dir == 0 ? __shfl_up(sc, 1, 64) : __shfl_down(sc, 1, 64);
        const float ex = dir == 0 ? (lane > 0 ? ex0 : 0.f) : (lane < 63 ? ex0 : 0.f);
        s0[qq] = dir == 0 ? ex + x0[qq] : ex + tot;
        s1[qq] = dir == 0 ? ex + tot : ex + x1[qq];
      }
      // the child of this lane: prefix [0, x) reads the sums at x - 1, suffix [x, n) at x
      int tq = 0;
      bool cv = false;
      const int gc = dir * SR_CM + (lane < SR_CM ? lane : 0);
      if (lane < SR_CM && crow(0)[gc] >= 2.f) {
        tq = dir == 0 ? XL[lane] - 1 : XR[lane];
        cv = true;
      }
      float v3[3];
#pragma unroll
      for (int qq = 0; qq < 3; ++qq) {
        const float a0v = __shfl(s0[qq], tq >> 1, 64), a1v = __shfl(s1[qq], tq >> 1, 64);
        v3[qq] = (tq & 1) ? a1v : a0v;
      }
      if (cv) {
        const float nch = crow(0)[gc], sr = crow(1)[gc];
        const float beta = dm.beta_frac * sr * (1.0f / nch);
        const float iden = 1.0f / (sr + nch * beta + dm.eps);
        crow(5)[gc] = (v3[0] + beta * (2.f * v3[1] + beta * v3[2])) * (iden * iden);
        crow(6)[gc] = beta;
        crow(7)[gc] = iden;
      }
    }
    __syncthreads();

    // ---- distortions of every child and probe (eq:app_node_and_drop_distortion).
    // With Y_t = sum G_tt' e_t' over t' < t (prefix children) or t' > t (suffix
    // children), the sums over a child of the increments
    //   e_t (Z), e_t (Y_t + u_t) (||M||^2), R_t u_t + e_t a_t and u_t + e_t g_t
    //   (<M, sum R v> and <M, sum v>), u_t = Y_t + e_t G_tt,
    // give Z_q, ||M_q||^2 and <M_q, v~> exactly as the sums over the child's token
    // pairs; the sums over each child are taken on the matrix cores with the
    // child masks (fp32 increments in three bf16 parts: exact products).  Y
    // comes from the Gram tiles and e (both in three parts; the three part
    // products below 2^-24 of |G e| are left out). ----
    if (probes) {
#pragma unroll 1
      for (int dir = 0; dir < 2; ++dir) {
        const float* av = sAG + 2 * dir * NMAX;
        const float* gv = av + NMAX;
        const u32x2 dmk = dir == 0 ? mlo : mup;
        int cl[2], ch[2];
        row_bounds(dir, cl[0], ch[0]);
        row_bounds(dir + 1, cl[1], ch[1]);
        f32x4 aZ[2], aS[2], aP[2], aQ[2];
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          aZ[c] = f32x4{0.f, 0.f, 0.f, 0.f}; aS[c] = aZ[c]; aP[c] = aZ[c]; aQ[c] = aZ[c];
        }
        // Y of a token tile from the Gram tiles in pairs (j2, j2 + 1) on the
        // 16x16x32 instruction: its operands take tile j2's four values of the
        // lane, then tile j2 + 1's (the A and B sides pair the tokens alike); a
        // half that must not contribute gets a zero Gram part, and e is zero
        // past the last tile
        static_assert(NTM % 2 == 0, "token tiles in pairs");
        auto cat = [](u32x2 a, u32x2 b) { return pk8(make_uint4(a.x, a.y, b.x, b.y)); };
#pragma unroll
        for (int i = 0; i < NTM; ++i) {
          if (i < nt) {
            f32x4 Y = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int j2 = 0; j2 < NTM; j2 += 2) {
              const bool use0 = j2 < nt && (j2 == i || (j2 < i ? dir == 0 : dir == 1));
              const bool use1 = j2 + 1 < nt && (j2 + 1 == i || (j2 + 1 < i ? dir == 0 : dir == 1));
              if (use0 || use1) {
                const u32x2 z2 = {0u, 0u};
                u32x2 gh0 = z2, gm0 = z2, gl0 = z2, gh1 = z2, gm1 = z2, gl1 = z2;
                if (use0) {
                  gread(i, j2, gh0, gm0, gl0);
                  if (j2 == i) { gh0 = gh0 & dmk; gm0 = gm0 & dmk; gl0 = gl0 & dmk; }
                }
                if (use1) {
                  gread(i, j2 + 1, gh1, gm1, gl1);
                  if (j2 + 1 == i) { gh1 = gh1 & dmk; gm1 = gm1 & dmk; gl1 = gl1 & dmk; }
                }
                const s16x8 ah = cat(gh0, gh1), am = cat(gm0, gm1), al = cat(gl0, gl1);
                const s16x8 bh = cat(eh[j2], eh[j2 + 1]), bm = cat(em[j2], em[j2 + 1]), bl = cat(el[j2], el[j2 + 1]);
                Y = mfma_bf16_16x16x32(al, bh, Y);
                Y = mfma_bf16_16x16x32(am, bm, Y);
                Y = mfma_bf16_16x16x32(ah, bl, Y);
                Y = mfma_bf16_16x16x32(am, bh, Y);
                Y = mfma_bf16_16x16x32(ah, bm, Y);
                Y = mfma_bf16_16x16x32(ah, bh, Y);
              }
            }
            const int t0 = 16 * i + 4 * g4;
            const float4 R4 = *(const float4*)(sR + t0), A4 = *(const float4*)(av + t0);
            const float4 G4 = *(const float4*)(gv + t0), D4 = *(const float4*)(sGd + t0);
            const float Rv[4] = {R4.x, R4.y, R4.z, R4.w}, Av[4] = {A4.x, A4.y, A4.z, A4.w};
            const float Gv[4] = {G4.x, G4.y, G4.z, G4.w}, Dg[4] = {D4.x, D4.y, D4.z, D4.w};
            // e_t = hi + mid + lo exactly
            float ev[4];
            {
              const uint32_t hv[4] = {eh[i].x << 16, eh[i].x & 0xffff0000u, eh[i].y << 16, eh[i].y & 0xffff0000u};
              const uint32_t mv[4] = {em[i].x << 16, em[i].x & 0xffff0000u, em[i].y << 16, em[i].y & 0xffff0000u};
              const uint32_t lv[4] = {el[i].x << 16, el[i].x & 0xffff0000u, el[i].y << 16, el[i].y & 0xffff0000u};
#pragma unroll
              for (int r = 0; r < 4; ++r) ev[r] = (__uint_as_float(hv[r]) + __uint_as_float(mv[r])) + __uint_as_float(lv[r]);
            }
            float xS[4], xP[4], xQ[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool ok = t0 + r < n;
              const float e = ev[r];
              const float u = Y[r] + e * Dg[r];
              xS[r] = ok ? e * (Y[r] + u) : 0.f;
              xP[r] = ok ? Rv[r] * u + e * Av[r] : 0.f;
              xQ[r] = ok ? u + e * Gv[r] : 0.f;
            }
            u32x2 sh, sm, sl, ph, pm, pl, qh, qm, ql;
            sr_split3(xS, sh, sm, sl);
            sr_split3(xP, ph, pm, pl);
            sr_split3(xQ, qh, qm, ql);
#pragma unroll
            for (int c = 0; c < 2; ++c) {
              const s16x4 mk = sr_op(one2 & mask16(cl[c], ch[c], t0));
              aZ[c] = mfma_bf16_16x16x16(mk, sr_op(el[i]), aZ[c]);
              aZ[c] = mfma_bf16_16x16x16(mk, sr_op(em[i]), aZ[c]);
              aZ[c] = mfma_bf16_16x16x16(mk, sr_op(eh[i]), aZ[c]);
              aS[c] = mfma_bf16_16x16x16(mk, sr_op(sl), aS[c]);
              aS[c] = mfma_bf16_16x16x16(mk, sr_op(sm), aS[c]);
              aS[c] = mfma_bf16_16x16x16(mk, sr_op(sh), aS[c]);
              aP[c] = mfma_bf16_16x16x16(mk, sr_op(pl), aP[c]);
              aP[c] = mfma_bf16_16x16x16(mk, sr_op(pm), aP[c]);
              aP[c] = mfma_bf16_16x16x16(mk, sr_op(ph), aP[c]);
              aQ[c] = mfma_bf16_16x16x16(mk, sr_op(ql), aQ[c]);
              aQ[c] = mfma_bf16_16x16x16(mk, sr_op(qm), aQ[c]);
              aQ[c] = mfma_bf16_16x16x16(mk, sr_op(qh), aQ[c]);
            }
          }
        }
        // lane (probe i16, g4) holds children 16 (dir + c) + 4 g4 + r:
        // ||M - z v~||^2 = ||M||^2 - 2 z <M, v~> + z^2 ||v~||^2 (clamped at 0)
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int ct = dir + c;
            const int gr = 16 * ct + 4 * g4 + r;
            const bool live = dir == 0 ? gr < nl : (gr >= SR_CM && gr - SR_CM < nr);
            const int grr = live ? gr : 0;
            const bool sc = live && crow(0)[grr] >= 2.f;
            const float z = ct == 0 ? zreg[0][r] : (ct == 1 ? zreg[1][r] : zreg[CT - 1][r]);
            const float Zs = aZ[c][r], s2 = aS[c][r];
            const float xv = (aP[c][r] + crow(6)[grr] * aQ[c][r]) * crow(7)[grr];
            const float s1 = fmaxf(s2 - 2.f * z * xv + z * z * crow(5)[grr], 0.f);
            const float dz = Zs - z;
            const float Dq = dm.lam_Z * dz * dz * __builtin_amdgcn_rcpf(Zs * Zs + dm.eps) +
                             dm.lam_M * s1 * __builtin_amdgcn_rcpf(s2 + dm.eps);
            const float con = row_sum16((sc && pok) ? (Zs * izc) * Dq : 0.f);
            if (sc && i16 == 0) sCon[gr * 4 + pt] = con;
          }
      }
    }
    __syncthreads();
    // D of each child: mean over the probes (fixed order)
    if (tid < nl + nr) {
      const int gc = tid < nl ? tid : SR_CM + (tid - nl);
      float acc = 0.f;
      if ((int)crow(0)[gc] >= 2) {
        for (int p4 = 0; p4 < 4 && 16 * p4 < dm.W; ++p4) acc += sCon[gc * 4 + p4];
        acc /= (float)dm.W;
      }
      crow(4)[gc] = acc;
    }
    __syncthreads();
    // ---- decision (fp32): best binary cut (smaller cut wins ties), then extraction ----
    if (wave == 0) {
      const float* cD = crow(4);
      const float* cRr = crow(1);
      const float kmn = __int_as_float(meta[4]), kmx = __int_as_float(meta[5]);
      const float kr = kmx - kmn;
      float best = -INFINITY;
      int bk = 0x7fffffff;
      if (lane < nb) {
        const int x = XB[lane];
        const float kh = kr > 0.f ? (sKap[x - 1] - kmn) / kr : 0.f;
        best = ((Dv - cD[posL[lane]]) - cD[SR_CM + posR[lane]]) + dm.lam_kappa * kh;
        bk = lane;
      }
      wave_argmax(best, bk);
      if (lane == 0) {
        const int iL = meta[6], iR = meta[7];
        float dsum = 0.f;
        int nkid = 1;
        if (p > 0) { dsum += cD[iL]; ++nkid; }
        if (p + 1 < n) { dsum += cD[SR_CM + iR]; ++nkid; }
        const float gext = (Dv - dsum) / (float)(nkid - 1);
        int ka[3], kn[3];
        float kD[3], kR[3];
        if (best >= gext) {
          const int bx = XB[bk];
          ka[0] = 0; kn[0] = bx; kD[0] = cD[posL[bk]]; kR[0] = cRr[posL[bk]];
          ka[1] = bx; kn[1] = n - bx; kD[1] = cD[SR_CM + posR[bk]]; kR[1] = cRr[SR_CM + posR[bk]];
          write_tree(1, bx, 2, ka, kn, kD, kR);
        } else {
          int c = 0;
          if (p > 0) { ka[c] = 0; kn[c] = p; kD[c] = cD[iL]; kR[c] = cRr[iL]; ++c; }
          ka[c] = p; kn[c] = 1; kD[c] = 0.f; kR[c] = sR[p]; ++c;
          if (p + 1 < n) { ka[c] = p + 1; kn[c] = n - p - 1; kD[c] = cD[SR_CM + iR]; kR[c] = cRr[SR_CM + iR]; ++c; }
          write_tree(2, p, c, ka, kn, kD, kR);
        }
      }
    }
    } while (0);
    publish_next();
  }
}

static hipError_t launch_split(const Dims& dm, int mode, int lvl, const void* K, const void* V, const void* Q,
                               const float* cosT, const float* sinT, const int32_t* slot_starts,
                               const int32_t* n_slots, const float* kappa, const TreeView& tv, int grid,
                               hipStream_t st) {
  const int lds = split_root_lds_bytes(dm.d);
  const Dims* dmp = (const Dims*)tv.kargs;
  const TreeView* tvp = (const TreeView*)((const char*)tv.kargs + 512);
#define GKV_SR(DD)                                                                                        \
  do {                                                                                                    \
    auto fn = (mode == BUILD_LEVEL || mode == BUILD_LEVEL_FULL) ? k_split_root<DD, true> : k_split_root<DD, false>; \
    hipError_t e0 = hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds); \
    if (e0 != hipSuccess) return e0;                                                                      \
    hipLaunchKernelGGL(fn, dim3(grid), dim3(SR_T), lds, st, dmp, mode, lvl, (const uint16_t*)K,           \
                       (const uint16_t*)V, (const uint16_t*)Q, cosT, sinT, slot_starts, n_slots, kappa, tvp); \
  } while (0)
  if (dm.d == 128) GKV_SR(128); else if (dm.d == 64) GKV_SR(64); else return hipErrorInvalidValue;
#undef GKV_SR
  return hipGetLastError();
}

hipError_t launch_split_root(const Dims& dm, int mode, const void* K, const void* V, const void* Q, const float* cosT,
                             const float* sinT, const int32_t* slot_starts, const int32_t* n_slots, const float* kappa,
                             const TreeView& tv, int grid, hipStream_t st) {
  return launch_split(dm, mode, 0, K, V, Q, cosT, sinT, slot_starts, n_slots, kappa, tv, grid, st);
}

hipError_t launch_split_level(const Dims& dm, bool full, int lvl, const void* K, const void* V, const void* Q,
                              const float* cosT, const float* sinT, const int32_t* slot_starts,
                              const int32_t* n_slots, const float* kappa, const TreeView& tv, int grid,
                              hipStream_t st) {
  return launch_split(dm, full ? BUILD_LEVEL_FULL : BUILD_LEVEL, lvl, K, V, Q, cosT, sinT, slot_starts, n_slots,
                      kappa, tv, grid, st);
}

}  // namespace gkv
