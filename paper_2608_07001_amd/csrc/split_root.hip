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
//     tokens of child c (prefix [0, x) or suffix [x, n)), alone or times R_t;
//     the B operand is k° = RoPE^{-1}(k) (staged in fp32 one half of the
//     dimensions at a time, the pair (i, i + d/2) rotated together), V^T (bf16)
//     or (R_t, ||k°_t||); fp32 operands go in three bf16 parts, so every
//     product is exact and only the fp32 accumulation rounds;
//   * child keys k~ = RoPE(mean k°, p), coherence, multiplicity, then
//     z = m_eff exp(k~ . q / sqrt(d) - m_q) for every child and probe on the
//     matrix cores (k~ split in three bf16 parts: exact products), held in
//     registers in the layout the scoring reads;
//   * distortion sweeps: wave = probe tile; it recomputes the probe
//     exponentials of each 16-token block (transposed logits on the matrix
//     cores), accumulates M^T = V^T E^T piece by piece between cuts with the
//     exact three-part split of e, and scores each child when the sweep
//     reaches its cut; prefix children left to right, then suffix children
//     right to left.  Cut positions are read into scalar registers, so the
//     sweep's control flow is uniform.  The value term of D_q is formed as
//     ||M||^2 - 2 z <M, v~> + z^2 ||v~||^2 (clamped at 0): its rounding error
//     is a few fp32 ulps of ||M||^2, i.e. about 1e-6 of the node's attention
//     mass in D, far below the distortions compared;
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
  static constexpr int LDV = NMAX + 8;                    // V^T row stride (bf16)
  static constexpr int KTS = D + 4;                       // child key row stride (fp32)
  static constexpr int KOB = NMAX * (H2 + 4) * 4;         // one half of k° [NMAX][H2 + 4] fp32
  static constexpr int VTB = D * LDV * 2;                 // V^T [D][LDV] bf16
  static constexpr int oX = 0;                            // k° half, then V^T
  static constexpr int oKt = (KOB > VTB ? KOB : VTB);     // [SR_CC][KTS] child k° sums -> k~
  static constexpr int oVv = oKt + SR_CC * KTS * 4;       // [SR_CC][D] v~
  static constexpr int oCs = oVv + SR_CC * D * 4;         // [6][SR_CC] n, sum R, mean ||k°||, m_eff, D, ||v~||^2
  static constexpr int oCon = oCs + 6 * SR_CC * 4;        // [SR_CC][4] per-wave D partials
  static constexpr int oPart = oCon + SR_CC * 4 * 4;      // [2][SR_CC][D/16] partial norms, [SR_CC][8] sums
  static constexpr int oR = oPart + (2 * (D / 16) + 8) * SR_CC * 4;   // [NMAX] R_t
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

template <int D>
__global__ __launch_bounds__(SR_T, 2) void k_split_root(const Dims* __restrict__ dmp, int mode,
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
  constexpr int DT = D / 16;               // 16-wide value tiles of M^T
  constexpr int CT = (SR_CC + 15) / 16;    // 16-wide child tiles
  extern __shared__ __align__(16) char smem[];
  float* sKo = (float*)(smem + Lay::oX);
  uint16_t* sVt = (uint16_t*)(smem + Lay::oX);
  float* sKt = (float*)(smem + Lay::oKt);
  float* sVv = (float*)(smem + Lay::oVv);
  float* sCs = (float*)(smem + Lay::oCs);
  float* sCon = (float*)(smem + Lay::oCon);
  float* sPart = (float*)(smem + Lay::oPart);
  float* sR = (float*)(smem + Lay::oR);
  float* sA = (float*)(smem + Lay::oA);
  float* sKap = (float*)(smem + Lay::oKap);
  float* sKn = (float*)(smem + Lay::oKn);
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
  const int nwork = tv.wctr[0];
  const float scale = 1.0f / sqrtf((float)D);
  const float LOG2E = 1.44269504088896341f;

  if (tid0 == 0) meta[9] = atomicAdd(&tv.wctr[1], 1);
  for (;;) {
    // per-lane indices are formed inside the loop (values derived from them are
    // not held across items, which would not fit the register budget)
    int tid = tid0;
    asm volatile("" : "+v"(tid));
    const int wave = uni(tid >> 6), lane = tid & 63, i16 = lane & 15, g4 = lane >> 4;
    const int pt = wave;                     // probe tile of this wave
    const int q = 16 * pt + i16;             // the lane's probe (scoring layout)
    const bool pok = q < dm.W;
    __syncthreads();
    const int wi = uni(meta[9]);
    __syncthreads();
    if (wi >= nwork) break;
    // the next item, in flight while this one is processed (stored before the
    // barrier at the top of the next pass)
    int wnext = 0;
    if (tid == 0) wnext = atomicAdd(&tv.wctr[1], 1);
    auto publish_next = [&]() { if (tid == 0) meta[9] = wnext; };
    do {
    // the work item: unit, slot, the root's D and R, w and the Add key (one load)
    const int4 d0 = *(const int4*)(tv.work + 8 * (int64_t)wi);
    const int4 d1 = *(const int4*)(tv.work + 8 * (int64_t)wi + 4);
    const int64_t unit = uni(d0.x);
    const int lg = (int)(unit / dm.J_cap), j = (int)(unit % dm.J_cap);
    const int l = lg / dm.G, g = lg % dm.G;
    const int a0 = uni(d0.y);
    const int n = uni(d0.z);
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
    // ---- writes the root and its children (local positions) ----
    auto write_tree = [&](int kind, int cut, int nkid, const int* ka, const int* kn, const float* kD,
                          const float* kR) {
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
    constexpr int CPR = D / 8;
    constexpr int VPT = (NMAX / 2) * CPR / SR_T;         // value items (token pair, 8-dim chunk) per thread
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
    float* sPvs = sPart + SR_CC * NP;        // [SR_CC][NP] ||v~||^2 partials
    float* sTmp = sPart + 2 * SR_CC * NP;    // [SR_CC][8] sum R and sum ||k°|| in three parts each
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
      // rotated together); every load of the half in flight first
      uint32_t kw1[IPT][4], kw2[IPT][4];
      float cs[IPT][8], sn[IPT][8];
#pragma unroll
      for (int it = 0; it < IPT; ++it) {
        const int e = tid + SR_T * it;
        const int ee = e < n * CH ? e : 0;
        const int t = ee / CH, c = 8 * (ee % CH);
        const int64_t ta = a0 + t;
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
        for (int s = 0; s < nks; ++s) {
          const int t0 = 16 * s + 4 * g4;
          float x[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) x[r] = t0 + r < n ? sKo[(t0 + r) * KSTR + 16 * tile + i16] : 0.f;
          u32x2 kh, km, kl;
          sr_split3(x, kh, km, kl);
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) {
            const s16x4 mk = sr_op(one2 & mask16(clo[ct], chi[ct], t0));
            acc[ct] = mfma_bf16_16x16x16(mk, sr_op(kl), acc[ct]);
            acc[ct] = mfma_bf16_16x16x16(mk, sr_op(km), acc[ct]);
            acc[ct] = mfma_bf16_16x16x16(mk, sr_op(kh), acc[ct]);
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

    // ---- value sums: V^T replaces k° ----
    {
      uint4 vraw[VPT][2];
#pragma unroll
      for (int it = 0; it < VPT; ++it) {             // every load in flight before the first store
        const int e = tid + SR_T * it;
        const int grp = e / (8 * CPR), rem = e % (8 * CPR);
        const int c = rem / 8, t = 2 * (8 * grp + rem % 8);
        vraw[it][0] = t < n ? *(const uint4*)(Vp + (int64_t)t * D + 8 * c) : make_uint4(0, 0, 0, 0);
        vraw[it][1] = t + 1 < n ? *(const uint4*)(Vp + (int64_t)(t + 1) * D + 8 * c) : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int it = 0; it < VPT; ++it) {
        const int e = tid + SR_T * it;
        const int grp = e / (8 * CPR), rem = e % (8 * CPR);
        const int c = rem / 8, t = 2 * (8 * grp + rem % 8);
        const uint4 v0 = vraw[it][0], v1 = vraw[it][1];
        const uint32_t pa[4] = {v0.x, v0.y, v0.z, v0.w}, pb[4] = {v1.x, v1.y, v1.z, v1.w};
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          *(uint32_t*)(sVt + (8 * c + 2 * h) * Lay::LDV + t) = (pa[h] & 0xffffu) | (pb[h] << 16);
          *(uint32_t*)(sVt + (8 * c + 2 * h + 1) * Lay::LDV + t) = (pa[h] >> 16) | (pb[h] & 0xffff0000u);
        }
      }
      if (tid < n) sKn[tid] = sqrtf(sKn[tid]);
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
        if (gr < SR_CC && i16 < 6) sTmp[gr * 8 + i16] = acc[r];
      }
    }
    __syncthreads();
    if (tid < SR_CC) {
      const float* x = sTmp + tid * 8;
      const float nch = crow(0)[tid];
      crow(1)[tid] = x[2] + x[1] + x[0];
      crow(2)[tid] = nch > 0.f ? (x[5] + x[4] + x[3]) / nch : 0.f;
    }
    __syncthreads();
    // wave = 16-dim value tiles: sum v and sum R v of every child, then v~
    // (eq:app_value_prototype) and the partial of ||v~||^2 over the tile
    for (int dt = wave; dt < DT; dt += SR_T / 64) {
      int clo[CT], chi[CT];
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) row_bounds(ct, clo[ct], chi[ct]);
      f32x4 av[CT], arv[CT];
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) { av[ct] = f32x4{0.f, 0.f, 0.f, 0.f}; arv[ct] = av[ct]; }
      for (int s = 0; s < nks; ++s) {
        const int t0 = 16 * s + 4 * g4;
        const uint2 vv = *(const uint2*)(sVt + (16 * dt + i16) * Lay::LDV + t0);
        u32x2 vb;
        vb.x = vv.x;
        vb.y = vv.y;
        const float4 r4 = *(const float4*)(sR + t0);
        const float rx[4] = {t0 < n ? r4.x : 0.f, t0 + 1 < n ? r4.y : 0.f, t0 + 2 < n ? r4.z : 0.f,
                             t0 + 3 < n ? r4.w : 0.f};
        u32x2 rh, rm, rl;
        sr_split3(rx, rh, rm, rl);
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
          const u32x2 mk = mask16(clo[ct], chi[ct], t0);
          av[ct] = mfma_bf16_16x16x16(sr_op(one2 & mk), sr_op(vb), av[ct]);
          arv[ct] = mfma_bf16_16x16x16(sr_op(rl & mk), sr_op(vb), arv[ct]);
          arv[ct] = mfma_bf16_16x16x16(sr_op(rm & mk), sr_op(vb), arv[ct]);
          arv[ct] = mfma_bf16_16x16x16(sr_op(rh & mk), sr_op(vb), arv[ct]);
        }
      }
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int gr = 16 * ct + 4 * g4 + r;
          const int grr = gr < SR_CC ? gr : 0;
          const float nch = crow(0)[grr];
          float vt = 0.f;
          if (nch >= 2.f) {
            const float sr = crow(1)[grr];
            const float beta = dm.beta_frac * sr * (1.0f / nch);
            vt = (arv[ct][r] + beta * av[ct][r]) / (sr + nch * beta + dm.eps);
          }
          const float ps = row_sum16(vt * vt);
          if (gr < SR_CC && nch >= 2.f) {
            sVv[gr * D + 16 * dt + i16] = vt;
            if (i16 == 0) sPvs[gr * NP + dt] = ps;
          }
        }
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
        float ss = 0.f, vs = 0.f;
#pragma unroll
        for (int k = 0; k < NP; ++k) { ss += sPss[tid * NP + k]; vs += sPvs[tid * NP + k]; }
        const float coh = sqrtf(ss) / (crow(2)[tid] + dm.eps);
        crow(3)[tid] = fminf(fmaxf(nch * coh * coh, 1.0f), nch);
        crow(5)[tid] = vs;
      }
    }
    {
      constexpr int RPT = (SR_CC * H2 + SR_T - 1) / SR_T;   // (child, pair) items per thread
      float ccv[RPT], snv[RPT];
#pragma unroll
      for (int m = 0; m < RPT; ++m) {         // the rotation rows, every load in flight together
        const int e = tid + SR_T * m;
        const int gc = e / H2, i = e % H2;
        int64_t pp = a0;
        if (e < SR_CC * H2) {
          const int nch = (int)crow(0)[gc];
          if (nch >= 2) {
            const int x0 = gc < SR_CM ? 0 : XR[gc - SR_CM];
            pp = round_half_even_mid(a0 + x0, a0 + x0 + nch);
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
    __syncthreads();

    // the first sweep's first key block (the prefix sweep's, or the suffix
    // sweep's when there is no prefix child), in flight during the z products
    uint32_t kcur[QW];
    {
      int tr = (nl > 0 ? 0 : 16 * ((n - 1) >> 4)) + i16;
      tr = tr < n ? tr : n - 1;
      const uint4* k4 = (const uint4*)(Kp + (int64_t)tr * D + QE * g4);
#pragma unroll
      for (int h = 0; h < QW / 4; ++h) {
        const uint4 v = k4[h];
        kcur[4 * h] = v.x; kcur[4 * h + 1] = v.y; kcur[4 * h + 2] = v.z; kcur[4 * h + 3] = v.w;
      }
    }
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

    // z moves to LDS in the scoring layout [child][probe], over the child key
    // rows (no longer read once every wave has its z)
    __syncthreads();
    float* sZt = sKt;
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int gr = 16 * ct + 4 * g4 + r;
        if (gr < SR_CC) sZt[gr * WMAX + q] = zreg[ct][r];
      }
    // ---- distortion sweeps: prefix children left to right, suffix children right to left ----
    // The sweep walks 16-token blocks; a block's probe exponentials and value
    // operands are formed once, then the pieces between the cuts inside it
    // are accumulated and each child is scored at its cut.
    if (16 * pt < dm.W) {
      const float sc2 = scale * LOG2E;
      for (int dir = 0; dir < 2; ++dir) {
        const bool prefix = dir == 0;
        const int nx = prefix ? nl : nr;
        if (nx == 0) continue;
        f32x4 M[DT];
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) M[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
        float Z = 0.f;
        int ci = prefix ? 0 : nx - 1;            // next cut (scalar)
        int cur = prefix ? 0 : n;                // tokens between 0 and cur (prefix) or cur and n (suffix) are in M
        for (int blk = prefix ? 0 : ((n - 1) >> 4); ; blk += prefix ? 1 : -1) {
          const int B0 = 16 * blk, B1 = min(B0 + 16, n);
          // the next key block in flight: the next block of this direction, or,
          // when every remaining cut lies in this block, the suffix sweep's first
          uint32_t knext[QW];
          {
            const bool last = prefix ? uni(XL[nx - 1]) <= B1 : uni(XR[0]) >= B0;
            const int nb2 = last ? (prefix ? ((n - 1) >> 4) : 0) : blk + (prefix ? 1 : -1);
            int tr = 16 * nb2 + i16;
            tr = tr < n ? tr : n - 1;
            const uint4* k4 = (const uint4*)(Kp + (int64_t)tr * D + QE * g4);
#pragma unroll
            for (int h = 0; h < QW / 4; ++h) {
              const uint4 v = k4[h];
              knext[4 * h] = v.x; knext[4 * h + 1] = v.y; knext[4 * h + 2] = v.z; knext[4 * h + 3] = v.w;
            }
          }
          // e_{q,t} of the block: transposed logits, lane holds tokens B0 + 4 g4 + r
          float ev[4];
          {
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < QE / 8; ++s)
              acc = mfma_bf16_16x16x32(pk8(make_uint4(kcur[4 * s], kcur[4 * s + 1], kcur[4 * s + 2], kcur[4 * s + 3])),
                                       pk8(make_uint4(qreg[4 * s], qreg[4 * s + 1], qreg[4 * s + 2], qreg[4 * s + 3])),
                                       acc);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int t = B0 + 4 * g4 + r;
              ev[r] = (pok && t < n) ? __builtin_amdgcn_exp2f(acc[r] * sc2 - mq2) : 0.f;
            }
          }
#pragma unroll
          for (int h = 0; h < QW; ++h) kcur[h] = knext[h];
          u32x2 eh, em, el;
          sr_split3(ev, eh, em, el);
          u32x2 vop[DT];
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            const uint2 vv = *(const uint2*)(sVt + (16 * dt + i16) * Lay::LDV + B0 + 4 * g4);
            vop[dt].x = vv.x;
            vop[dt].y = vv.y;
          }
          const int t0 = B0 + 4 * g4;
          bool more = true;
          for (;;) {
            const int x = uni(prefix ? XL[ci] : XR[ci]);
            const bool inblk = prefix ? (x <= B1) : (x >= B0);
            const int pend = inblk ? x : (prefix ? B1 : B0);
            const int lo = prefix ? cur : pend, hi = prefix ? pend : cur;
            if (hi > lo) {                       // the piece [lo, hi) of this block
              bool in[4];
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                in[r] = (unsigned)(t0 + r - lo) < (unsigned)(hi - lo);
                Z += in[r] ? ev[r] : 0.f;
              }
              u32x2 mk;
              mk.x = (in[0] ? 0xffffu : 0u) | (in[1] ? 0xffff0000u : 0u);
              mk.y = (in[2] ? 0xffffu : 0u) | (in[3] ? 0xffff0000u : 0u);
              const s16x4 ph = sr_op(eh & mk), pm = sr_op(em & mk), pl = sr_op(el & mk);
#pragma unroll
              for (int dt = 0; dt < DT; ++dt) {
                const s16x4 va = sr_op(vop[dt]);
                M[dt] = mfma_bf16_16x16x16(va, pl, M[dt]);
                M[dt] = mfma_bf16_16x16x16(va, pm, M[dt]);
                M[dt] = mfma_bf16_16x16x16(va, ph, M[dt]);
              }
            }
            cur = pend;
            if (!inblk) break;
            // child gc at cut x: z of the lane's probe from the lane holding row gc % 16
            const int gc = prefix ? ci : SR_CM + ci;
            const int nch = prefix ? x : n - x;
            if (nch >= 2) {
              const float z = sZt[gc * WMAX + q];
              // ||M - z v~||^2 = ||M||^2 - 2 z <M, v~> + z^2 ||v~||^2
              float s2a = 0.f, s2b = 0.f, xva = 0.f, xvb = 0.f;
              const float* vv = sVv + gc * D + 4 * g4;
#pragma unroll
              for (int dt = 0; dt < DT; ++dt) {
                const float4 v4 = *(const float4*)(vv + 16 * dt);
                const float vt[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                  const float Mv = M[dt][r];
                  if (dt & 1) { s2b += Mv * Mv; xvb += Mv * vt[r]; }
                  else { s2a += Mv * Mv; xva += Mv * vt[r]; }
                }
              }
              const float s2 = col_sum4(s2a + s2b);
              const float xv = col_sum4(xva + xvb);
              const float Zs = col_sum4(Z);
              const float s1 = fmaxf(s2 - 2.f * z * xv + z * z * crow(5)[gc], 0.f);
              const float dz = Zs - z;
              const float Dq = dm.lam_Z * dz * dz * __builtin_amdgcn_rcpf(Zs * Zs + dm.eps) +
                               dm.lam_M * s1 * __builtin_amdgcn_rcpf(s2 + dm.eps);
              const float con = row_sum16((g4 == 0 && pok) ? (Zs * izc) * Dq : 0.f);
              if (lane == 0) sCon[gc * 4 + pt] = con;
            }
            ci += prefix ? 1 : -1;
            if (prefix ? ci >= nx : ci < 0) { more = false; break; }
          }
          if (!more) break;
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

hipError_t launch_split_root(const Dims& dm, int mode, const void* K, const void* V, const void* Q, const float* cosT,
                             const float* sinT, const int32_t* slot_starts, const int32_t* n_slots, const float* kappa,
                             const TreeView& tv, int grid, hipStream_t st) {
  const int lds = split_root_lds_bytes(dm.d);
  const Dims* dmp = (const Dims*)tv.kargs;
  const TreeView* tvp = (const TreeView*)((const char*)tv.kargs + 512);
#define GKV_SR(DD)                                                                                        \
  do {                                                                                                    \
    auto fn = k_split_root<DD>;                                                                           \
    hipError_t e0 = hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds); \
    if (e0 != hipSuccess) return e0;                                                                      \
    hipLaunchKernelGGL(fn, dim3(grid), dim3(SR_T), lds, st, dmp, mode, (const uint16_t*)K,                \
                       (const uint16_t*)V, (const uint16_t*)Q, cosT, sinT, slot_starts, n_slots, kappa, tvp); \
  } while (0)
  if (dm.d == 128) GKV_SR(128); else if (dm.d == 64) GKV_SR(64); else return hipErrorInvalidValue;
#undef GKV_SR
  return hipGetLastError();
}

}  // namespace gkv
