// Root evaluation of every (layer, KV head, slot) unit, bf16 caches.
//
// Same outputs as the fp32 root kernel (root.hip): pass 2 of the direct
// relevance R_t (App. A.4 eq:app_attention_probability, eq:app_direct_relevance),
// the probe exponentials e_{q,t} and probe masses A_t (App. A.3 "Prototype
// distortion"), the root prototype (eq:app_rope_prototype, eq:app_value_prototype,
// eq:app_effective_multiplicity), its distortion D and D_drop
// (eq:app_original_attention_stats .. eq:app_node_and_drop_distortion) and the
// key of the unit's Add operation (App. A.5 eq:app_operation_gains,
// eq:app_unit_utility).
//
// Work layout.  A workgroup of 4 waves walks a contiguous range of units
// (layer/head-major, so consecutive units share Q); wave w owns the window
// queries [16w, 16w + 16) with every query head of the group, their Q rows held
// in registers.  Tokens go in blocks of 32 through the 16x16x32 bf16
// instruction:
//   * logits come out transposed (tokens x queries, one token tile of 16 per
//     output tile), so lane (query i, group g) holds tokens 4g .. 4g + 3 of
//     each of the block's two tiles;
//   * those eight probe exponentials are the lane's B operand of
//     M^T = V^T E^T for the whole block: the contraction runs over the block's
//     tokens in the order (g, tile, r), and V^T is staged in LDS with its
//     token columns permuted the same way, so the A operand is one 16-byte
//     read; e is split into three bf16 parts (exact products);
//   * per unit, four workgroup barriers: staging done, token loop done, token
//     values done, prototype done (one thread per dimension of k~ and v~);
//     every wave then finishes its probes' distortions on its own, and the
//     unit's outputs are written after the next unit's staging barrier.  LDS
//     stays under 80 KB, so two workgroups share a CU.
#include "common.h"

namespace gkv {

constexpr int RB_T = 256;          // threads per workgroup
constexpr int RB_W = RB_T / 64;    // waves
constexpr int RB_GRID = 2048;      // persistent workgroups (two per CU, four rounds)
constexpr int RB_GRID_RI = 4096;   // ... without K rows in LDS (four per CU, four rounds)

// RI: the token relevance pass ran before (no relevance partials, no K rows).
// The prototype k~, v~ share the probe-mass partials' space: those are last
// read before barrier B, the prototype is first written after it and last read
// before the next unit's barrier S.
template <int D, bool RI>
struct RbLds {
  static constexpr int LDK = D + 8;          // K rows [NMAX][LDK] bf16
  static constexpr int LDV = NMAX + 8;       // V^T rows [D][LDV] bf16, token columns permuted per 32-block
  static constexpr int oVt = 0;
  static constexpr int oRp = oVt + D * LDV * 2;             // [RB_W][NMAX] relevance partials (not RI)
  static constexpr int oAp = oRp + (RI ? 0 : RB_W * NMAX * 4);   // [RB_W][NMAX] probe-mass partials
  static constexpr int oKt = oAp;                           // [D] prototype key k~
  static constexpr int oVv = oKt + D * 4;                   // [D] prototype value v~
  static constexpr int oKp = oVv + D * 4;                   // [3][D] k~ in three bf16 parts
  static_assert(2 * D * 4 + 3 * D * 2 <= RB_W * NMAX * 4, "prototype inside the probe-mass partials");
  static constexpr int oR = oAp + RB_W * NMAX * 4;          // [NMAX] R_t
  static constexpr int oA = oR + NMAX * 4;                  // [NMAX] A_t
  static constexpr int oKn = oA + NMAX * 4;                 // [NMAX] ||k°_t||
  static constexpr int oPk = oKn + NMAX * 4;                // [RB_W][D] partial sums of the turned keys
  static constexpr int oSum = oPk + RB_W * D * 4;           // [RB_W][4] per-wave sums of R, A, ||k°||
  static constexpr int oRed = oSum + RB_W * 4 * 4;          // [2][RB_W] distortion sums (unit parity)
  static constexpr int oPend = oRed + 2 * RB_W * 4;         // deferred outputs of the previous unit
  static constexpr int oK = oPend + 64;                     // K rows [NMAX][LDK] (not RI)
  static constexpr int bytes = RI ? oK : oK + NMAX * LDK * 2;
};

int root_bf16_lds_bytes(int d) { return d == 128 ? RbLds<128, false>::bytes : RbLds<64, false>::bytes; }

// LDS column of token t of a unit: within each 32-token block, the token
// 16 h + 4 g + r (tile h, lane group g, row r) sits at 8 g + 4 h + r
__device__ __forceinline__ int perm32(int t) {
  return (t & ~31) | ((t & 12) << 1) | ((t >> 2) & 4) | (t & 3);
}

// e = hi + mid + lo exactly, each a bf16: hi keeps the top 8 significant bits
// of e (truncation), mid the next 8, lo the last 8 (exact in bf16).  Eight
// values packed two per 32-bit word in k order.
__device__ __forceinline__ void split3x8(const float* e, uint4& hi, uint4& mid, uint4& lo) {
  uint32_t h[8], m[8], l[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    h[r] = __float_as_uint(e[r]) & 0xffff0000u;
    const float r1 = e[r] - __uint_as_float(h[r]);
    m[r] = __float_as_uint(r1) & 0xffff0000u;
    l[r] = __float_as_uint(r1 - __uint_as_float(m[r]));
  }
  // upper halves of two words: bytes 2, 3 of the first and 2, 3 of the second
#define GKV_HI2(a, b) __builtin_amdgcn_perm((b), (a), 0x07060302u)
  hi = make_uint4(GKV_HI2(h[0], h[1]), GKV_HI2(h[2], h[3]), GKV_HI2(h[4], h[5]), GKV_HI2(h[6], h[7]));
  mid = make_uint4(GKV_HI2(m[0], m[1]), GKV_HI2(m[2], m[3]), GKV_HI2(m[4], m[5]), GKV_HI2(m[6], m[7]));
  lo = make_uint4(GKV_HI2(l[0], l[1]), GKV_HI2(l[2], l[3]), GKV_HI2(l[4], l[5]), GKV_HI2(l[6], l[7]));
#undef GKV_HI2
}

__device__ __forceinline__ float pick4f(const float* v, int i) {
  return i == 0 ? v[0] : i == 1 ? v[1] : i == 2 ? v[2] : v[3];
}

// RI: the direct relevance s-hat is already in the token values (the token
// relevance pass ran before), so only the probe rows are evaluated here.
template <int D, bool MP, bool RI>
__global__ __launch_bounds__(RB_T, RI ? 4 : 2) void k_root_bf(const Dims* __restrict__ dmp, const uint16_t* __restrict__ K,
                                                     const uint16_t* __restrict__ V, const uint16_t* __restrict__ Q,
                                                     const float* __restrict__ cosT, const float* __restrict__ sinT,
                                                     const int32_t* __restrict__ slot_starts,
                                                     const int32_t* __restrict__ n_slots, const TreeView* __restrict__ tvp) {
  // the argument structures are read from device memory where used (held in
  // scalar registers they would not fit)
  const Dims& dm = *dmp;
  const TreeView& tv = *tvp;
  using Lay = RbLds<D, RI>;
  constexpr int H2 = D / 2;
  constexpr int DT = D / 16;                 // 16-wide value tiles of M^T
  constexpr int KS = D / 32;                 // k steps of a logit tile
  constexpr int HG = RI ? 1 : 4;             // head slots whose Q rows are held at once
  constexpr int CHP = H2 / 8;                // 8-dim pair chunks per token in the k° staging
  constexpr int CPR = D / 8;                 // 16-byte chunks per V row
  extern __shared__ __align__(16) char smem[];
  uint16_t* sVt = (uint16_t*)(smem + Lay::oVt);
  uint16_t* sK = (uint16_t*)(smem + Lay::oK);
  float* sRp = (float*)(smem + Lay::oRp);
  float* sAp = (float*)(smem + Lay::oAp);
  float* sKn = (float*)(smem + Lay::oKn);
  float* sR = (float*)(smem + Lay::oR);
  float* sA = (float*)(smem + Lay::oA);
  float* sPk = (float*)(smem + Lay::oPk);
  float* sKt = (float*)(smem + Lay::oKt);
  float* sVv = (float*)(smem + Lay::oVv);
  uint16_t* sKp = (uint16_t*)(smem + Lay::oKp);
  float* sSum = (float*)(smem + Lay::oSum);
  float* sRed = (float*)(smem + Lay::oRed);

  const int tid0 = threadIdx.x, w = tid0 >> 6;
  const int J = *n_slots;
  if (J < 1 || J > dm.J_cap) {                // malformed partition: nothing to build
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(tv.status, STATUS_PARTITION);
    return;
  }
  const int64_t total = (int64_t)dm.L * dm.G * J;
  const int64_t per = (total + gridDim.x - 1) / gridDim.x;
  const int64_t ub = (int64_t)blockIdx.x * per;
  const int64_t ue = ub + per < total ? ub + per : total;
  const float scale = 1.0f / sqrtf((float)D);
  const float sc2 = scale * 1.44269504088896341f;   // logit scale in base-2 exponent units
  const int lane0 = tid0 & 63;
  const int u = 16 * w + (lane0 & 15);        // the lane's window query
  const bool uok = u < dm.W;
  const int uq = uok ? u : 0;
  const int hp = uq % dm.hpg;                 // query head of probe u
  const bool wave_on = 16 * w < dm.W;
  const bool wave_full = 16 * w + 16 <= dm.W;  // every query of the wave exists
  const int npass = (MP && !RI) ? (dm.hpg + HG - 1) / HG : 1;
  const int klast = HG * (npass - 1);         // first slot of the last pass (run first)
  // Q rows of head slots k0 .. k0 + HG - 1 (slot k = head (hp + k) mod |H(g)|): lane (i, g)
  // holds dims 32 s + 8 g .. + 7 of its query for k step s; row statistics (m_V, 1 / Z_V),
  // weight 0 for a slot past |H(g)|
  uint4 qr[HG][KS];
  float cR[HG];                               // log2 of e^{m_V} Z_V (+inf: slot past |H(g)|)
  float mq2 = 0.f, zcq = 1.f;                 // probe shift m_q log2(e) and 1 / Z_q(C)
  float Sg = 1.f, om = 0.f;
  int cur_lg = -1;
  auto load_pass = [&](int l, int g, int lg, int k0) {
    const int g8 = (lane0 >> 4) * 8;
#pragma unroll
    for (int h = 0; h < HG; ++h) {
      const int k = k0 + h;
      const int hl = (hp + k) % dm.hpg;
      const uint16_t* qrow = Q + (((int64_t)l * dm.H + (int64_t)g * dm.hpg + hl) * dm.W + uq) * D;
#pragma unroll
      for (int s = 0; s < KS; ++s) qr[h][s] = *(const uint4*)(qrow + 32 * s + g8);
      if constexpr (!RI) {
        const float4 st = tv.row_stats[(int64_t)lg * dm.rows + hl * dm.W + uq];
        cR[h] = k < dm.hpg ? st.x * 1.44269504088896341f + __log2f(st.y) : INFINITY;
      }
    }
  };

  // deferred outputs of the previous unit: written and read by thread 0 only,
  // kept in LDS (not registers) across the next unit's staging
  struct Pend { int64_t unit, sl; int n, a0; uint32_t ord; float sr, dd, om; };
  static_assert(sizeof(Pend) <= 64, "deferred-output record");
  Pend* sP = (Pend*)(smem + Lay::oPend);
  bool pend = false;
  auto flush = [&](int buf) {
    const Pend P = *sP;
    const int64_t p_unit = P.unit, p_sl = P.sl;
    const int p_n = P.n, p_a0 = P.a0;
    const uint32_t p_ord = P.ord;
    const float p_sr = P.sr, p_dd = P.dd, p_om = P.om;
    float Dv = 0.f;
#pragma unroll
    for (int w2 = 0; w2 < RB_W; ++w2) Dv += sRed[buf * RB_W + w2];
    Dv = p_n >= 2 ? Dv / (float)dm.W : 0.f;
    tv.node_a[p_sl] = p_a0;
    tv.node_n[p_sl] = p_n;
    tv.node_child[p_sl] = -1;
    tv.node_parent[p_sl] = -1;
    tv.node_nch[p_sl] = 0;
    tv.node_kind[p_sl] = 0;
    tv.node_cut[p_sl] = -1;
    tv.node_D[p_sl] = Dv;
    tv.node_R[p_sl] = p_sr;
    tv.unit_nn[p_unit] = 1;
    tv.unit_Ddrop[p_unit] = p_dd;
    const float Ua = utility(add_gain(p_om, p_sr, p_dd, Dv), 1);
    tv.add_U[p_unit] = Ua;
    tv.add_E[p_unit] = op_key(Ua, p_ord * 256u);
    tv.add_exec[p_unit] = 0;
  };

  int buf = 0;
  // (layer, KV head, slot) of the unit, stepped along the range (no division per unit)
  int lg = (int)(ub / J), j = (int)(ub % J);
  int l = lg / dm.G, g = lg % dm.G;
  for (int64_t uu = ub; uu < ue; ++uu, ++j) {
    if (j == J) {
      j = 0;
      ++lg;
      if (++g == dm.G) { g = 0; ++l; }
    }
    // per-thread addresses are formed inside the loop (not held across it)
    int tid = tid0;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63, i16 = lane & 15, g4 = lane >> 4;
    const int64_t unit = (int64_t)lg * dm.J_cap + j;
    const int64_t a0 = slot_starts[j];
    const int n = slot_starts[j + 1] - (int)a0;
    if (n < 1 || n > NMAX || a0 < 0 || a0 + n > dm.N_c) {   // malformed partition: refuse the unit
      if (tid == 0) { atomicOr(tv.status, STATUS_PARTITION); tv.unit_nn[unit] = 0; }
      continue;
    }
    const int nb = (n + 31) >> 5;             // 32-token blocks
    const uint16_t* Kp = K + ((int64_t)lg * dm.T + a0) * D;
    const uint16_t* Vp = V + ((int64_t)lg * dm.T + a0) * D;
    if (lg != cur_lg || (MP && !RI)) {
      if (wave_on) load_pass(l, g, lg, klast);
      if (lg != cur_lg) {
        if (wave_on) {
          mq2 = tv.probe_m[(int64_t)lg * dm.W + uq] * 1.44269504088896341f;
          zcq = 1.0f / tv.probe_ZC[(int64_t)lg * dm.W + uq];
        }
        Sg = tv.lg_S[lg] + dm.eps;
        om = tv.omega[lg];
        cur_lg = lg;
      }
    }
    const int64_t pmid = round_half_even_mid((int)a0, (int)a0 + n);
    float* Kn = sKn;

    // ---- staging: K rows (zero past n) turned to the representative position
    // on the way (R_{p~} R_{p_t}^{-1} is the turn by p~ - p_t) for the k~ sums
    // and ||k°_t||; V^T with permuted token columns (zero past n) ----
    float kacc[16];                           // partial sums of the turned keys (written after barrier S)
    const int c = 8 * (tid % CHP);
    {
#pragma unroll
      for (int h = 0; h < 16; ++h) kacc[h] = 0.f;
      // K item e: token e / CHP, pair chunk c (rows up to n; not RI: up to 32 nb, zero past n);
      // V item e: token pair 16 (e / (16 CPR)) + e % 16 (pairs fastest within a
      // 32-token block), 8-dim chunk (e / 16) % CPR.  One item of each kind per
      // thread and round, all its loads issued before any is used (a second
      // round in flight would not fit the register budget).
      const int nk = (RI ? n : 32 * nb) * CHP, nv = 16 * nb * CPR;
      const int nmax = nk > nv ? nk : nv;
      for (int e = tid; e < nmax; e += RB_T) {
        const int t = e / CHP;
        const int tk = t < n ? t : n - 1;
        const uint4 k1 = *(const uint4*)(Kp + (int64_t)tk * D + c);
        const uint4 k2 = *(const uint4*)(Kp + (int64_t)tk * D + c + H2);
        // the turn from position a0 + tk to the representative position is
        // the table row of their distance, its sine negated for a token past it
        const int dl = (int)(a0 + tk - pmid);
        const int64_t ta = dl < 0 ? -dl : dl;
        const uint32_t sgn = dl < 0 ? 0x80000000u : 0u;
        const float4 c0 = *(const float4*)(cosT + ta * H2 + c), c1 = *(const float4*)(cosT + ta * H2 + c + 4);
        const float4 s0 = *(const float4*)(sinT + ta * H2 + c), s1 = *(const float4*)(sinT + ta * H2 + c + 4);
        const int cv = (e / 16) % CPR, t0 = 2 * (16 * (e / (16 * CPR)) + e % 16);
        const int ta0 = t0 < n ? t0 : n - 1, ta1 = t0 + 1 < n ? t0 + 1 : n - 1;
        const uint4 v0 = *(const uint4*)(Vp + (int64_t)ta0 * D + 8 * cv);
        const uint4 v1 = *(const uint4*)(Vp + (int64_t)ta1 * D + 8 * cv);
        if (e < nk) {
          uint4 ka = k1, kc = k2;
          if (t >= n) { ka = make_uint4(0, 0, 0, 0); kc = ka; }
          if constexpr (!RI) {                // RI: the logits read K from L2 (staged here once)
            *(uint4*)(sK + t * Lay::LDK + c) = ka;
            *(uint4*)(sK + t * Lay::LDK + c + H2) = kc;
          }
          const uint32_t w1[4] = {ka.x, ka.y, ka.z, ka.w}, w2[4] = {kc.x, kc.y, kc.z, kc.w};
          const float cs8[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
          const float sn8[8] = {__uint_as_float(__float_as_uint(s0.x) ^ sgn), __uint_as_float(__float_as_uint(s0.y) ^ sgn),
                                __uint_as_float(__float_as_uint(s0.z) ^ sgn), __uint_as_float(__float_as_uint(s0.w) ^ sgn),
                                __uint_as_float(__float_as_uint(s1.x) ^ sgn), __uint_as_float(__float_as_uint(s1.y) ^ sgn),
                                __uint_as_float(__float_as_uint(s1.z) ^ sgn), __uint_as_float(__float_as_uint(s1.w) ^ sgn)};
          // the pair (a1, a2) turned, added in place; ||k°_t||^2 from the key
          // itself (a turn keeps the norm)
          float ss = 0.f;
#pragma unroll
          for (int h = 0; h < 8; ++h) {
            const float a1 = __uint_as_float((h & 1) ? (w1[h >> 1] & 0xffff0000u) : (w1[h >> 1] << 16));
            const float a2 = __uint_as_float((h & 1) ? (w2[h >> 1] & 0xffff0000u) : (w2[h >> 1] << 16));
            kacc[h] = fmaf(a1, cs8[h], fmaf(a2, sn8[h], kacc[h]));
            kacc[8 + h] = fmaf(a2, cs8[h], fmaf(-a1, sn8[h], kacc[8 + h]));
            ss = fmaf(a1, a1, fmaf(a2, a2, ss));
          }
#pragma unroll
          for (int o = 1; o < CHP; o <<= 1) ss += __shfl_xor(ss, o, 64);
          if (t < n && c == 0) Kn[t] = sqrtf(ss);
        }
        if (e < nv) {
          uint4 va = v0, vb = v1;
          if (t0 >= n) va = make_uint4(0, 0, 0, 0);
          if (t0 + 1 >= n) vb = make_uint4(0, 0, 0, 0);
          const uint32_t pa[4] = {va.x, va.y, va.z, va.w}, pb[4] = {vb.x, vb.y, vb.z, vb.w};
          const int col = perm32(t0);          // t0 even: t0 + 1 sits at col + 1
#pragma unroll
          for (int h = 0; h < 4; ++h) {
            *(uint32_t*)(sVt + (8 * cv + 2 * h) * Lay::LDV + col) = (pa[h] & 0xffffu) | (pb[h] << 16);
            *(uint32_t*)(sVt + (8 * cv + 2 * h + 1) * Lay::LDV + col) = (pa[h] >> 16) | (pb[h] & 0xffff0000u);
          }
        }
      }
      // lanes l, l + CHP, ... of a wave hold the same chunk
      static_assert(CHP == 4 || CHP == 8, "chunk classes within a 16-lane row");
      if constexpr (CHP == 8) {
        // eight lanes per chunk (lane bits 3, 4, 5): each exchange halves the
        // values a lane holds and doubles the lanes summed (lane ^ 8 by a DPP
        // rotation inside the row, then the row swaps of permlane16/32, which
        // leave the first operand's sum in the even rows (the lower half) and
        // the second's in the odd rows (upper half)); lane (chunk, b3 b4 b5)
        // ends with the chunk's values 8 b3 + 4 b4 + 2 b5 and one more
        const bool b3 = (lane >> 3) & 1;
        float r1[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float snd = b3 ? kacc[i] : kacc[8 + i], kp = b3 ? kacc[8 + i] : kacc[i];
          r1[i] = kp + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(snd), 0x128, 0xf, 0xf, false));
        }
        float r2[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const auto pq = __builtin_amdgcn_permlane16_swap(__float_as_uint(r1[i]), __float_as_uint(r1[i + 4]), false, false);
          r2[i] = __uint_as_float(pq[0]) + __uint_as_float(pq[1]);
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const auto pq = __builtin_amdgcn_permlane32_swap(__float_as_uint(r2[i]), __float_as_uint(r2[i + 2]), false, false);
          kacc[i] = __uint_as_float(pq[0]) + __uint_as_float(pq[1]);
        }
      } else {
        // rotations by 4 and 8 within each 16-lane row (DPP), then the row swaps
#pragma unroll
        for (int h = 0; h < 16; ++h) {
          float v = kacc[h];
          v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x124, 0xf, 0xf, false));
          v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xf, 0xf, false));
          kacc[h] = col_sum4(v);
        }
      }
      // empty Split slots of the unit's node range: cost 0 (the flat scans
      // over the ops read a slot's key only where its cost is not 0; the
      // refinement writes every field of a node it creates, the scoring pass
      // every field of a live node, the selection every execution flag)
      static_assert(NMAX <= RB_T, "one thread per slot pair");
      uint16_t* spc = (uint16_t*)(tv.sp_cost + ((int64_t)lg * dm.N_c + a0) * 2);
      if (tid < n) spc[tid] = 0;
    }
    __syncthreads();                          // S: staging done; every wave is past the previous unit
    if (tid == 0 && pend) flush(buf ^ 1);
    if constexpr (CHP == 8) {
      const int h0 = 8 * ((lane >> 3) & 1) + 4 * ((lane >> 4) & 1) + 2 * ((lane >> 5) & 1);
      const int dd = h0 < 8 ? c + h0 : c + H2 + (h0 - 8);
      *(float2*)(sPk + w * D + dd) = make_float2(kacc[0], kacc[1]);
    } else if (lane < CHP) {
#pragma unroll
      for (int h = 0; h < 8; ++h) { sPk[w * D + c + h] = kacc[h]; sPk[w * D + c + H2 + h] = kacc[8 + h]; }
    }

    // ---- token loop: logits, relevance partials, probe exponentials, M^T ----
    f32x4 Macc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) Macc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float Zl = 0.f;
    if (wave_on) {
      for (int k0 = klast; k0 >= 0; k0 -= HG) {
        if (MP && !RI && k0 != klast) load_pass(l, g, lg, k0);
        for (int b = 0; b < nb; ++b) {
          float ev[8];                        // probe exponentials of the block, (tile, row) order
          const bool full = wave_full && 32 * b + 32 <= n;   // no token or query to mask
          // RI: the block's K fragments straight from L2 (the rows were just
          // read by the staging), rows past n clamped (their logits are masked)
          uint4 kg[RI ? 2 : 1][KS];
          if constexpr (RI) {
#pragma unroll
            for (int tl = 0; tl < 2; ++tl) {
              const int tr = 32 * b + 16 * tl + i16;
              const uint16_t* kr = Kp + (int64_t)(tr < n ? tr : n - 1) * D + 8 * g4;
#pragma unroll
              for (int s = 0; s < KS; ++s) kg[tl][s] = *(const uint4*)(kr + 32 * s);
            }
          }
#pragma unroll
          for (int tl = 0; tl < 2; ++tl) {
            const int t0 = 32 * b + 16 * tl + 4 * g4;   // the lane's first token of this tile
            f32x4 acc[HG];
#pragma unroll
            for (int h = 0; h < HG; ++h) acc[h] = f32x4{0.f, 0.f, 0.f, 0.f};
            {
              uint4 kv[KS];
              if constexpr (RI) {
#pragma unroll
                for (int s = 0; s < KS; ++s) kv[s] = kg[tl][s];
              } else {
                const uint16_t* kr = sK + (32 * b + 16 * tl + i16) * Lay::LDK + 8 * g4;
#pragma unroll
                for (int s = 0; s < KS; ++s) kv[s] = *(const uint4*)(kr + 32 * s);
              }
#pragma unroll
              for (int s = 0; s < KS; ++s)
#pragma unroll
                for (int h = 0; h < HG; ++h) acc[h] = mfma_bf16_16x16x32(pk8(kv[s]), pk8(qr[h][s]), acc[h]);
            }
            // lane holds tokens t0 + r of its query in every slot:
            // pi = e^{l - m_V} / Z_V = 2^(acc sc2 - cR)
            float Rp[4];
            if constexpr (!RI) {
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                float s = 0.f;
#pragma unroll
                for (int h = 0; h < HG; ++h) s += __builtin_amdgcn_exp2f(acc[h][r] * sc2 - cR[h]);
                Rp[r] = (full || (uok && t0 + r < n)) ? s : 0.f;
              }
            }
            if (k0 == 0) {
              float ap[4];
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                // exp2(-inf) = 0 for the masked ones: no branch around the exponential
                const float e = __builtin_amdgcn_exp2f((full || (uok && t0 + r < n)) ? acc[0][r] * sc2 - mq2 : -INFINITY);
                ev[4 * tl + r] = e;
                ap[r] = e * zcq;
                Zl += e;
              }
#pragma unroll
              for (int r = 0; r < 4; ++r) ap[r] = row_sum16(ap[r]);
              if (i16 < 4) sAp[w * NMAX + t0 + i16] = pick4f(ap, i16);
            }
            if constexpr (!RI) {
#pragma unroll
              for (int r = 0; r < 4; ++r) Rp[r] = row_sum16(Rp[r]);
              if (i16 < 4) {
                float* dst = sRp + w * NMAX + t0 + i16;
                *dst = (k0 == klast ? 0.f : *dst) + pick4f(Rp, i16);
              }
            }
          }
          if (k0 == 0) {
            uint4 eh, em, el;
            split3x8(ev, eh, em, el);
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
              const s16x8 va = pk8(*(const uint4*)(sVt + (16 * dt + i16) * Lay::LDV + 32 * b + 8 * g4));
              Macc[dt] = mfma_bf16_16x16x32(va, pk8(el), Macc[dt]);
              Macc[dt] = mfma_bf16_16x16x32(va, pk8(em), Macc[dt]);
              Macc[dt] = mfma_bf16_16x16x32(va, pk8(eh), Macc[dt]);
            }
          }
        }
      }
    }
    __syncthreads();                          // A: token loop done

    // ---- token values R_t, A_t (LDS and out, zero up to 32 nb) and their sums ----
    {
      float R = 0.f, A = 0.f, kn = 0.f;
      if (tid < n) {
        float s = 0.f, am = 0.f;
#pragma unroll
        for (int w2 = 0; w2 < RB_W; ++w2)
          if (16 * w2 < dm.W) {
            if constexpr (!RI) s += sRp[w2 * NMAX + tid];
            am += sAp[w2 * NMAX + tid];
          }
        if constexpr (RI) R = tv.tok_R[(int64_t)lg * dm.N_c + a0 + tid];
        else R = s / Sg;
        if (tv.dhat) R = (1.f - dm.lam_graph) * R + dm.lam_graph * tv.dhat[a0 + tid];   // eq:app_bottom_up_value
        A = am / (float)dm.W;
        kn = Kn[tid];
        tv.tok_R[(int64_t)lg * dm.N_c + a0 + tid] = R;
        tv.tok_A[(int64_t)lg * dm.N_c + a0 + tid] = A;
      }
      if (tid < 32 * nb) { sR[tid] = R; sA[tid] = A; }
      R = wave_sum_dpp(R);
      A = wave_sum_dpp(A);
      kn = wave_sum_dpp(kn);
      if (lane == 0) { sSum[4 * w] = R; sSum[4 * w + 1] = A; sSum[4 * w + 2] = kn; }
    }
    __syncthreads();                          // B: token values and their sums in LDS
    const float sr = sSum[0] + sSum[4] + sSum[8] + sSum[12];
    const float inv = 1.0f / (float)n;
    if (tid < D) {
      // v~ of dim tid: sums of R v and v over the unit, four tokens per step (a
      // column quad of V^T holds consecutive tokens)
      const int d = tid;
      float vr = 0.f, vs = 0.f;
      for (int q = 0; q < 8 * nb; ++q) {
        const int col = 4 * q;
        const int t0 = (col & ~31) | ((col & 4) << 2) | ((col >> 1) & 12);
        const uint2 vw = *(const uint2*)(sVt + d * Lay::LDV + col);
        const float4 r4 = *(const float4*)(sR + t0);
        const float v4[4] = {__uint_as_float(vw.x << 16), __uint_as_float(vw.x & 0xffff0000u),
                             __uint_as_float(vw.y << 16), __uint_as_float(vw.y & 0xffff0000u)};
        vr += r4.x * v4[0] + r4.y * v4[1] + r4.z * v4[2] + r4.w * v4[3];
        vs += (v4[0] + v4[1]) + (v4[2] + v4[3]);
      }
      const float beta = dm.beta_frac * sr * inv;
      sVv[d] = (vr + beta * vs) / (sr + (float)n * beta + dm.eps);
    } else if (tid < 2 * D) {
      // k~ of dim tid - D: the mean of the keys turned to the representative
      // position (the staging summed them turned there)
      const int d = tid - D;
      float m = 0.f;
#pragma unroll
      for (int q = 0; q < RB_W; ++q) m += sPk[q * D + d];
      const float kt = m * inv;
      sKt[d] = kt;
      // k~ = hi + mid + lo exactly (each a bf16) for the q . k~ products
      const uint32_t hb = __float_as_uint(kt) & 0xffff0000u;
      const float r1 = kt - __uint_as_float(hb);
      const uint32_t mb = __float_as_uint(r1) & 0xffff0000u;
      const uint32_t lb = __float_as_uint(r1 - __uint_as_float(mb));
      sKp[d] = (uint16_t)(hb >> 16);
      sKp[D + d] = (uint16_t)(mb >> 16);
      sKp[2 * D + d] = (uint16_t)(lb >> 16);
    }
    __syncthreads();                          // C: prototype in LDS
    if (tid < 2 * D) {                        // the unit's root prototype, as pack writes it
      uint16_t* pr = (uint16_t*)tv.proto + unit * 2 * D;
      pr[tid] = f32_to_bf16_rne(tid < D ? sKt[tid] : sVv[tid - D]);
    }

    // ---- this wave's probe distortions ----
    {
      const float sa = sSum[1] + sSum[5] + sSum[9] + sSum[13];
      const float skn = sSum[2] + sSum[6] + sSum[10] + sSum[14];
      // coherence of the mean k° (eq:app_effective_multiplicity); a turn keeps its norm
      float ss = 0.f;
      for (int d = lane; d < D; d += 64) {
        float m = 0.f;
#pragma unroll
        for (int q = 0; q < RB_W; ++q) m += sPk[q * D + d];
        m *= inv;
        ss += m * m;
      }
      ss = wave_sum_dpp(ss);
      const float coh = sqrtf(ss) / (skn * inv + dm.eps);
      const float me = fminf(fmaxf((float)n * coh * coh, 1.0f), (float)n);
      if (tid == 0) tv.proto_logm[unit] = logf(me);
      float con = 0.f;
      if (wave_on) {
        float vv = 0.f;                        // ||v~||^2
        for (int d = lane; d < D; d += 64) vv = fmaf(sVv[d], sVv[d], vv);
        vv = wave_sum_dpp(vv);
        // q . k~ for the wave's probes (head slot 0) on the matrix cores: A rows
        // 0-2 hold k~ in three bf16 parts (exact products), B the probes' query
        // rows; lane (probe, g4 = 0) gets the three parts and passes the sum on
        f32x4 qa = {0.f, 0.f, 0.f, 0.f};
        const uint16_t* kp = sKp + (i16 < 3 ? i16 : 0) * D + 8 * g4;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          uint4 a8 = *(const uint4*)(kp + 32 * s);
          if (i16 >= 3) a8 = make_uint4(0u, 0u, 0u, 0u);
          qa = mfma_bf16_16x16x32(pk8(a8), pk8(qr[0][s]), qa);
        }
        const float qk = __shfl((qa[0] + qa[1]) + qa[2], i16, 64);
        const float z = me * __builtin_amdgcn_exp2f(qk * sc2 - mq2);
        const float Z = col_sum4(Zl);
        // ||M - z v~||^2 = ||M||^2 - 2 z <M, v~> + z^2 ||v~||^2 (clamped at 0), as
        // the refinement forms it: a rounding error of a few fp32 ulps of ||M||^2
        float mv = 0.f, s2 = 0.f;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const float4 v4 = *(const float4*)(sVv + 16 * dt + 4 * g4);
          const float vt[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float M = Macc[dt][r];
            mv = fmaf(M, vt[r], mv);
            s2 = fmaf(M, M, s2);
          }
        }
        mv = col_sum4(mv);
        s2 = col_sum4(s2);
        const float s1 = fmaxf(s2 - 2.f * z * mv + z * z * vv, 0.f);
        const float dz = Z - z;
        const float Dq = dm.lam_Z * dz * dz * __builtin_amdgcn_rcpf(Z * Z + dm.eps) +
                         dm.lam_M * s1 * __builtin_amdgcn_rcpf(s2 + dm.eps);
        con = (uok && g4 == 0) ? (Z * zcq) * Dq : 0.f;
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) con += __shfl_xor(con, o, 64);
      }
      if (lane == 0) sRed[buf * RB_W + w] = con;
      if (tid == 0) {
        pend = true;
        Pend P;
        P.unit = unit;
        P.sl = (int64_t)lg * 2 * dm.N_c + 2 * a0;
        P.n = n;
        P.a0 = (int)a0;
        P.ord = (uint32_t)lg * (uint32_t)J + (uint32_t)j;
        P.sr = sr;
        P.dd = sa;
        P.om = om;
        *sP = P;
      }
    }
    buf ^= 1;
  }
  __syncthreads();
  if (tid0 == 0 && pend) flush(buf ^ 1);
}

hipError_t launch_root_bf16(const Dims& dm, const void* K, const void* V, const void* Q, const float* cosT,
                            const float* sinT, const int32_t* slot_starts, const int32_t* n_slots, const TreeView& tv,
                            hipStream_t st) {
  const int64_t cap = (int64_t)dm.L * dm.G * dm.J_cap;
  const bool ri = token_relevance_pass(dm);   // s-hat already in the token values
  // RI: no relevance partials and no K rows in LDS, four workgroups per CU
  const int64_t gmax = ri ? RB_GRID_RI : RB_GRID;
  const dim3 grid((unsigned)(cap < gmax ? cap : gmax));
  const int lds = ri ? (dm.d == 128 ? RbLds<128, true>::bytes : RbLds<64, true>::bytes) : root_bf16_lds_bytes(dm.d);
#define GKV_LAUNCH_ROOT_BF(DD)                                                                              \
  do {                                                                                                      \
    auto fn = ri ? k_root_bf<DD, false, true> : (dm.hpg > 4 ? k_root_bf<DD, true, false> : k_root_bf<DD, false, false>); \
    hipError_t e0 = hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds);  \
    if (e0 != hipSuccess) return e0;                                                                        \
    hipLaunchKernelGGL(fn, grid, dim3(RB_T), lds, st, (const Dims*)tv.kargs, (const uint16_t*)K,            \
                       (const uint16_t*)V, (const uint16_t*)Q, cosT, sinT, slot_starts, n_slots,               \
                       (const TreeView*)((const char*)tv.kargs + 512));                           \
  } while (0)
  if (dm.d == 128) GKV_LAUNCH_ROOT_BF(128); else if (dm.d == 64) GKV_LAUNCH_ROOT_BF(64);
  else return hipErrorInvalidValue;
#undef GKV_LAUNCH_ROOT_BF
  return hipGetLastError();
}

}  // namespace gkv
