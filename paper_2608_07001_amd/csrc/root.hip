// Root evaluation of every (layer, KV head, slot) unit.
//
// For each unit [a0, a0 + n) of one (l, g) this computes, in one pass over the
// unit's keys and values:
//   * pass 2 of the direct relevance (App. A.4 eq:app_attention_probability,
//     eq:app_direct_relevance): R_t = s-hat_t for each token, from the row
//     statistics of pass 1, or (1 - lambda_graph) s-hat_t + lambda_graph d-hat_t
//     when a multi-hop relevance is given (eq:app_bottom_up_value);
//   * the probe exponentials e_{q,t} = exp(l_{q,t} - m_q) of the distortion
//     probes (App. A.3 "Prototype distortion") and A_t, the probe-mean of
//     e_{q,t} / Z_q(C) (the attention mass a dropped token takes away);
//   * the root prototype (eq:app_rope_prototype, eq:app_value_prototype,
//     eq:app_effective_multiplicity), its distortion D (eq:app_original_attention_stats
//     .. eq:app_node_and_drop_distortion), D_drop and the key of the unit's Add
//     operation (App. A.5 eq:app_operation_gains, eq:app_unit_utility).
//
// Layout of the work.  A workgroup of 4 waves walks a contiguous range of units
// (layer/head-major, so consecutive units share Q).  Wave w owns the window
// queries u in [16w, 16w + 16) and, for each, every query head of the group:
// the logits of a 16-token block come out of the matrix cores transposed
// (tokens x queries), so each lane holds 4 tokens of one query.  In that layout
// the probe exponentials of the block are already the B operand of the next
// product M^T = V^T E^T (values x probes), which the matrix cores accumulate
// over the unit; e is split into three bf16 parts so the products are exact
// (fp32 data uses the fp32 matrix instruction directly).  The Q quarter rows of
// one head at a time is held in registers, the next one in flight.
#include "common.h"

namespace gkv {

constexpr int RT = 256;          // threads per workgroup
constexpr int RWV = RT / 64;     // waves: wave w owns window queries [16w, 16w + 16)
constexpr int ROOT_GRID = 2048;  // persistent workgroups (several rounds of 2 per CU)

template <typename T, int D>
struct RootLds {
  static constexpr bool BF = sizeof(T) == 2;
  static constexpr int LDK = BF ? D + 8 : D + 4;        // K rows [NMAX][LDK]
  static constexpr int LDV = BF ? NMAX + 8 : NMAX + 4;  // V^T rows [D][LDV]
  static constexpr int NPK = RWV;                       // per-wave partial sums of k°
  static constexpr int NPV = RT / D;                    // token phases of the v sums
  // V^T first and the small arrays next keep every fixed offset within the 16-bit
  // immediate of the LDS instructions; K rows are addressed per tile anyway
  static constexpr int oVt = 0;
  static constexpr int oRp = oVt + D * LDV * (int)sizeof(T);   // [RWV][NMAX] relevance partials
  static constexpr int oAp = oRp + RWV * NMAX * 4;              // [RWV][NMAX] probe-mass partials
  static constexpr int oR = oAp + RWV * NMAX * 4;               // [NMAX] R_t
  static constexpr int oA = oR + NMAX * 4;                      // [NMAX] A_t
  static constexpr int oKn = oA + NMAX * 4;                     // [NMAX] ||k_t||
  static constexpr int oPk = oKn + NMAX * 4;                    // [NPK][D] partial sums of k°
  static constexpr int oPv = oPk + NPK * D * 4;                 // [NPV][D] partial sums of R v
  static constexpr int oPs = oPv + NPV * D * 4;                 // [NPV][D] partial sums of v
  static constexpr int oKt = oPs + NPV * D * 4;                 // [D] prototype key k~
  static constexpr int oVv = oKt + D * 4;                       // [D] prototype value v~
  static constexpr int oRed = oVv + D * 4;                      // [16] unit scalars
  static constexpr int oK = oRed + 16 * 4;                      // K rows [NMAX][LDK]
  static constexpr int bytes = oK + NMAX * LDK * (int)sizeof(T);
};

int root_lds_bytes(const Dims& dm) {
  if (dm.dtype == GRACEKV_BF16) return root_bf16_lds_bytes(dm.d);
  return dm.d == 128 ? RootLds<float, 128>::bytes : RootLds<float, 64>::bytes;
}

__device__ __forceinline__ float pick4(const float* v, int i) {
  return i == 0 ? v[0] : i == 1 ? v[1] : i == 2 ? v[2] : v[3];
}
// bf16 of a finite value, round to nearest even
__device__ __forceinline__ uint32_t bf16_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}
// e = hi + mid + lo with each part a bf16 (the remainders are exact in fp32)
__device__ __forceinline__ void split3(const float* e, s16x4& hi, s16x4& mid, s16x4& lo) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const uint32_t h = bf16_bits(e[r]);
    const float r1 = e[r] - __uint_as_float(h << 16);
    const uint32_t m = bf16_bits(r1);
    const float r2 = r1 - __uint_as_float(m << 16);
    hi[r] = (short)h;
    mid[r] = (short)m;
    lo[r] = (short)bf16_bits(r2);
  }
}

// One 16-byte chunk of the staging of a unit: a K pair chunk (dims c .. c + 7
// and c + H2 .. c + H2 + 7 of token t) with its RoPE rows, and two V chunks
// (dims 8 cv .. 8 cv + 7 of tokens tv and tv + 1).  bf16 only.
struct StageChunk {
  uint4 k1, k2, v0, v1;
  float4 c0, c1, s0, s1;
};

template <typename T, int D, bool MP>
__global__ __launch_bounds__(RT, 2) void k_root(Dims dm, const T* __restrict__ K, const T* __restrict__ V,
                                                const T* __restrict__ Q, const float* __restrict__ cosT,
                                                const float* __restrict__ sinT, const int32_t* __restrict__ slot_starts,
                                                const int32_t* __restrict__ n_slots, TreeView tv) {
  using Lay = RootLds<T, D>;
  constexpr bool BF = Lay::BF;
  constexpr int H2 = D / 2;
  constexpr int DT = D / 16;                 // 16-wide value tiles of M^T
  constexpr int QE = D / 4;                  // elements of a lane's quarter row
  constexpr int QW = BF ? QE / 2 : QE;       // ... in 32-bit words
  constexpr int HG = 4;                      // head slots whose Q rows are held at once
  extern __shared__ __align__(16) char smem[];
  T* sK = (T*)(smem + Lay::oK);
  T* sVt = (T*)(smem + Lay::oVt);
  float* sRp = (float*)(smem + Lay::oRp);
  float* sAp = (float*)(smem + Lay::oAp);
  float* sR = (float*)(smem + Lay::oR);
  float* sA = (float*)(smem + Lay::oA);
  float* sKn = (float*)(smem + Lay::oKn);
  float* sPk = (float*)(smem + Lay::oPk);
  float* sPv = (float*)(smem + Lay::oPv);
  float* sPs = (float*)(smem + Lay::oPs);
  float* sKt = (float*)(smem + Lay::oKt);
  float* sVv = (float*)(smem + Lay::oVv);
  float* sRed = (float*)(smem + Lay::oRed);

  const int tid0 = threadIdx.x, w = tid0 >> 6, g4o = (tid0 >> 4) & 3;
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
  const int u = 16 * w + (tid0 & 15);         // the lane's window query
  const bool uok = u < dm.W;
  const int uq = uok ? u : 0;
  const int hp = uq % dm.hpg;                 // query head of probe u
  const bool wave_on = 16 * w < dm.W;
  // passes over the unit, HG head slots each (MP: more than one, so Q is reloaded per pass)
  const int npass = MP ? (dm.hpg + HG - 1) / HG : 1;
  const int klast = HG * (npass - 1);         // first slot of the last pass (run first)

  constexpr int CHP = H2 / 8;                // 8-dim pair chunks per token in the k° staging
  // Q quarter rows of head slots k0 .. k0 + HG - 1 (slot k = head (hp + k) mod |H(g)|) and
  // their row statistics (m_V, 1 / Z_V); a slot past |H(g)| gets weight 0.  With one pass
  // they stay valid for every unit of the same (l, g).
  uint32_t qr[HG][QW];
  float2 rs[HG];
  float mq = 0.f, zcq = 1.f;                  // probe shift and 1 / Z_q(C)
  float Sg = 1.f, om = 0.f;                   // S_{l,g} and the head weight of the current (l, g)
  int cur_lg = -1;
  auto load_pass = [&](int l, int g, int lg, int k0) {
#pragma unroll
    for (int h = 0; h < HG; ++h) {
      const int k = k0 + h;
      const int hl = (hp + k) % dm.hpg;
      const uint4* q4 = (const uint4*)(Q + (((int64_t)l * dm.H + (int64_t)g * dm.hpg + hl) * dm.W + uq) * D + QE * g4o);
#pragma unroll
      for (int x = 0; x < QW / 4; ++x) {
        const uint4 v = q4[x];
        qr[h][4 * x] = v.x; qr[h][4 * x + 1] = v.y; qr[h][4 * x + 2] = v.z; qr[h][4 * x + 3] = v.w;
      }
      const float4 st = tv.row_stats[(int64_t)lg * dm.rows + hl * dm.W + uq];
      rs[h] = make_float2(st.x, k < dm.hpg ? 1.0f / st.y : 0.f);
    }
  };

  for (int64_t uu = ub; uu < ue; ++uu) {
    // the thread index passes through an empty asm per unit, so that per-thread
    // addresses are formed inside the loop instead of being held in registers across it
    int tid = tid0;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63, i16 = lane & 15, g4 = lane >> 4;
    const int lg = (int)(uu / J), j = (int)(uu % J);
    const int l = lg / dm.G, g = lg % dm.G;
    const int64_t unit = (int64_t)lg * dm.J_cap + j;
    const int64_t a0 = slot_starts[j];
    const int n = slot_starts[j + 1] - (int)a0;
    if (n < 1 || n > NMAX || a0 < 0 || a0 + n > dm.N_c) {   // malformed partition: refuse the unit
      if (tid == 0) { atomicOr(tv.status, STATUS_PARTITION); tv.unit_nn[unit] = 0; }
      continue;
    }
    const int rows16 = (n + 15) & ~15;
    const int n_tt = rows16 / 16;
    const T* Kp = K + ((int64_t)lg * dm.T + a0) * D;
    const T* Vp = V + ((int64_t)lg * dm.T + a0) * D;
    if (lg != cur_lg || MP) {
      if (wave_on) load_pass(l, g, lg, klast);
      if (lg != cur_lg) {
        if (wave_on) {
          mq = tv.probe_m[(int64_t)lg * dm.W + uq];
          zcq = 1.0f / tv.probe_ZC[(int64_t)lg * dm.W + uq];
        }
        Sg = tv.lg_S[lg] + dm.eps;
        om = tv.omega[lg];
        cur_lg = lg;
      }
    }
    // representative position of the root and its RoPE row (wave 0, used at the end)
    const int64_t pmid = round_half_even_mid((int)a0, (int)a0 + n);
    float pcos = 0.f, psin = 0.f;
    if (w == 0) { pcos = cosT[pmid * H2 + (lane % H2)]; psin = sinT[pmid * H2 + (lane % H2)]; }
    __syncthreads();                          // the previous unit is done with LDS

    // ---- stage K (row-major) and undo RoPE on the way: per-thread sums of k°
    // for the thread's 8-dim pair chunk, ||k°_t|| reduced across the CHP lanes
    // of token t; V transposed; zero past n ----
    {
      float kacc[16];
#pragma unroll
      for (int h = 0; h < 16; ++h) kacc[h] = 0.f;
      const int c = 8 * (tid % CHP);
      // k°, ||k°|| and the partial sums of one token chunk (k1 holds dims c.., k2 dims c + H2..)
      auto rope_undo = [&](int t, const float* k1, const float* k2, const float* cs8, const float* sn8) {
        float ss = 0.f;
#pragma unroll
        for (int h = 0; h < 8; ++h) {
          const float o1 = k1[h] * cs8[h] + k2[h] * sn8[h];
          const float o2 = k2[h] * cs8[h] - k1[h] * sn8[h];
          kacc[h] += o1;
          kacc[8 + h] += o2;
          ss += o1 * o1 + o2 * o2;
        }
#pragma unroll
        for (int o = 1; o < CHP; o <<= 1) ss += __shfl_xor(ss, o, 64);
        if (t < n && c == 0) sKn[t] = sqrtf(ss);
      };
      if constexpr (BF) {
        constexpr int CPR = D / 8;            // 16-byte chunks per row of V
        const int cnt = rows16 * CHP;         // = (rows16 / 2) * CPR
        // every load is unconditional (rows clamped to the unit) so that the loads of two
        // chunks are in flight together; rows past n are zeroed after the load
        auto load = [&](int e) {
          StageChunk s;
          const int t = e / CHP;
          const int tk = t < n ? t : n - 1;
          const uint4* kp = (const uint4*)(Kp + (int64_t)tk * D + c);
          s.k1 = kp[0];
          s.k2 = *(const uint4*)(Kp + (int64_t)tk * D + c + H2);
          const int64_t ta = a0 + tk;
          s.c0 = *(const float4*)(cosT + ta * H2 + c); s.c1 = *(const float4*)(cosT + ta * H2 + c + 4);
          s.s0 = *(const float4*)(sinT + ta * H2 + c); s.s1 = *(const float4*)(sinT + ta * H2 + c + 4);
          const int grp = e / (8 * CPR), rem = e % (8 * CPR);
          const int cv = rem / 8, tv0 = 2 * (8 * grp + rem % 8);
          const int t0c = tv0 < n ? tv0 : n - 1, t1c = tv0 + 1 < n ? tv0 + 1 : n - 1;
          s.v0 = *(const uint4*)(Vp + (int64_t)t0c * D + 8 * cv);
          s.v1 = *(const uint4*)(Vp + (int64_t)t1c * D + 8 * cv);
          return s;
        };
        auto store = [&](int e, StageChunk s) {
          const int t = e / CHP;
          if (t >= n) { s.k1 = make_uint4(0, 0, 0, 0); s.k2 = s.k1; }
          *(uint4*)(sK + t * Lay::LDK + c) = s.k1;
          *(uint4*)(sK + t * Lay::LDK + c + H2) = s.k2;
          const uint32_t w1[4] = {s.k1.x, s.k1.y, s.k1.z, s.k1.w}, w2[4] = {s.k2.x, s.k2.y, s.k2.z, s.k2.w};
          float k1[8], k2[8];
#pragma unroll
          for (int h = 0; h < 4; ++h) {
            k1[2 * h] = __uint_as_float(w1[h] << 16); k1[2 * h + 1] = __uint_as_float(w1[h] & 0xffff0000u);
            k2[2 * h] = __uint_as_float(w2[h] << 16); k2[2 * h + 1] = __uint_as_float(w2[h] & 0xffff0000u);
          }
          const float cs8[8] = {s.c0.x, s.c0.y, s.c0.z, s.c0.w, s.c1.x, s.c1.y, s.c1.z, s.c1.w};
          const float sn8[8] = {s.s0.x, s.s0.y, s.s0.z, s.s0.w, s.s1.x, s.s1.y, s.s1.z, s.s1.w};
          rope_undo(t, k1, k2, cs8, sn8);
          const int grp = e / (8 * CPR), rem = e % (8 * CPR);
          const int cv = rem / 8, tv0 = 2 * (8 * grp + rem % 8);
          if (tv0 >= n) s.v0 = make_uint4(0, 0, 0, 0);
          if (tv0 + 1 >= n) s.v1 = make_uint4(0, 0, 0, 0);
          const uint32_t a[4] = {s.v0.x, s.v0.y, s.v0.z, s.v0.w}, b[4] = {s.v1.x, s.v1.y, s.v1.z, s.v1.w};
#pragma unroll
          for (int h = 0; h < 4; ++h) {
            *(uint32_t*)(sVt + (8 * cv + 2 * h) * Lay::LDV + tv0) = (a[h] & 0xffffu) | (b[h] << 16);
            *(uint32_t*)(sVt + (8 * cv + 2 * h + 1) * Lay::LDV + tv0) = (a[h] >> 16) | (b[h] & 0xffff0000u);
          }
        };
        for (int e = tid; e < cnt; e += RT) store(e, load(e));
      } else {
        for (int e = tid; e < rows16 * CHP; e += RT) {
          const int t = e / CHP;
          float k1[8], k2[8];
          float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a, cq = a, dq = a;
          if (t < n) {
            const float4* p1 = (const float4*)((const float*)Kp + (int64_t)t * D + c);
            const float4* p2 = (const float4*)((const float*)Kp + (int64_t)t * D + c + H2);
            a = p1[0]; b = p1[1]; cq = p2[0]; dq = p2[1];
          }
          float4* d1 = (float4*)((float*)sK + t * Lay::LDK + c);
          float4* d2 = (float4*)((float*)sK + t * Lay::LDK + c + H2);
          d1[0] = a; d1[1] = b; d2[0] = cq; d2[1] = dq;
          k1[0] = a.x; k1[1] = a.y; k1[2] = a.z; k1[3] = a.w; k1[4] = b.x; k1[5] = b.y; k1[6] = b.z; k1[7] = b.w;
          k2[0] = cq.x; k2[1] = cq.y; k2[2] = cq.z; k2[3] = cq.w; k2[4] = dq.x; k2[5] = dq.y; k2[6] = dq.z; k2[7] = dq.w;
          const int64_t ta = a0 + (t < n ? t : n - 1);
          const float4 c0 = *(const float4*)(cosT + ta * H2 + c), c1 = *(const float4*)(cosT + ta * H2 + c + 4);
          const float4 s0 = *(const float4*)(sinT + ta * H2 + c), s1 = *(const float4*)(sinT + ta * H2 + c + 4);
          const float cs8[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
          const float sn8[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
          rope_undo(t, k1, k2, cs8, sn8);
        }
        constexpr int CPR = D / 4;
        for (int e = tid; e < rows16 * CPR; e += RT) {
          const int grp = e / (16 * CPR), rem = e % (16 * CPR);
          const int cv = rem / 16, t = 16 * grp + rem % 16;
          float4 vv = make_float4(0.f, 0.f, 0.f, 0.f);
          if (t < n) vv = *(const float4*)(Vp + (int64_t)t * D + 4 * cv);
          sVt[(4 * cv + 0) * Lay::LDV + t] = vv.x;
          sVt[(4 * cv + 1) * Lay::LDV + t] = vv.y;
          sVt[(4 * cv + 2) * Lay::LDV + t] = vv.z;
          sVt[(4 * cv + 3) * Lay::LDV + t] = vv.w;
        }
      }
      // lanes l, l + CHP, ... of the wave hold the same chunk
#pragma unroll
      for (int o = CHP; o < 64; o <<= 1)
#pragma unroll
        for (int h = 0; h < 16; ++h) kacc[h] += __shfl_xor(kacc[h], o, 64);
      if (lane < CHP) {
#pragma unroll
        for (int h = 0; h < 8; ++h) { sPk[w * D + c + h] = kacc[h]; sPk[w * D + c + H2 + h] = kacc[8 + h]; }
      }
    }
    __syncthreads();

    // ---- logits, relevance, probe exponentials and M^T = V^T E^T: per 16-token
    // tile the HG held head slots together; the pass holding the probe head
    // (slot 0) runs last ----
    f32x4 Macc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) Macc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float Zl = 0.f;
    if (wave_on) {
      for (int k0 = klast; k0 >= 0; k0 -= HG) {
        if (MP && k0 != klast) load_pass(l, g, lg, k0);
        for (int tb = 0; tb < n_tt; ++tb) {
          const int t0 = 16 * tb;
          uint32_t kreg[QW];
          {
            const uint4* k4 = (const uint4*)(sK + (t0 + i16) * Lay::LDK + QE * g4);
#pragma unroll
            for (int x = 0; x < QW / 4; ++x) {
              const uint4 v = k4[x];
              kreg[4 * x] = v.x; kreg[4 * x + 1] = v.y; kreg[4 * x + 2] = v.z; kreg[4 * x + 3] = v.w;
            }
          }
          f32x4 acc[HG];
#pragma unroll
          for (int h = 0; h < HG; ++h) acc[h] = f32x4{0.f, 0.f, 0.f, 0.f};
          if constexpr (BF) {
#pragma unroll
            for (int s = 0; s < QE / 4; ++s)
#pragma unroll
              for (int h = 0; h < HG; ++h)
                acc[h] = mfma_bf16_16x16x16(pk4(kreg[2 * s], kreg[2 * s + 1]), pk4(qr[h][2 * s], qr[h][2 * s + 1]), acc[h]);
          } else {
#pragma unroll
            for (int s = 0; s < QE; ++s)
#pragma unroll
              for (int h = 0; h < HG; ++h)
                acc[h] = mfma_f32_16x16x4(__uint_as_float(kreg[s]), __uint_as_float(qr[h][s]), acc[h]);
          }
          // lane holds tokens t0 + 4 g4 + r of the lane's query row in every slot
          float Rp[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            float s = 0.f;
#pragma unroll
            for (int h = 0; h < HG; ++h) s += fexp(acc[h][r] * scale - rs[h].x) * rs[h].y;
            Rp[r] = (uok && t0 + 4 * g4 + r < n) ? s : 0.f;
          }
          if (k0 == 0) {
            float ev[4], ap[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              ev[r] = fexp((uok && t0 + 4 * g4 + r < n) ? acc[0][r] * scale - mq : -INFINITY);   // e^-inf = 0: no branch
              ap[r] = ev[r] * zcq;
              Zl += ev[r];
            }
            if constexpr (BF) {
              s16x4 eh, em, el;
              split3(ev, eh, em, el);
#pragma unroll
              for (int dt = 0; dt < DT; ++dt) {
                const uint2 vv = *(const uint2*)(sVt + (16 * dt + i16) * Lay::LDV + t0 + 4 * g4);
                const s16x4 va = pk4(vv.x, vv.y);
                Macc[dt] = mfma_bf16_16x16x16(va, el, Macc[dt]);
                Macc[dt] = mfma_bf16_16x16x16(va, em, Macc[dt]);
                Macc[dt] = mfma_bf16_16x16x16(va, eh, Macc[dt]);
              }
            } else {
#pragma unroll
              for (int dt = 0; dt < DT; ++dt) {
                const float4 vv = *(const float4*)(sVt + (16 * dt + i16) * Lay::LDV + t0 + 4 * g4);
                Macc[dt] = mfma_f32_16x16x4(vv.x, ev[0], Macc[dt]);
                Macc[dt] = mfma_f32_16x16x4(vv.y, ev[1], Macc[dt]);
                Macc[dt] = mfma_f32_16x16x4(vv.z, ev[2], Macc[dt]);
                Macc[dt] = mfma_f32_16x16x4(vv.w, ev[3], Macc[dt]);
              }
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) ap[r] = row_sum16(ap[r]);
            if (i16 < 4) sAp[w * NMAX + t0 + 4 * g4 + i16] = pick4(ap, i16);
          }
#pragma unroll
          for (int r = 0; r < 4; ++r) Rp[r] = row_sum16(Rp[r]);
          if (i16 < 4) {
            float* dst = sRp + w * NMAX + t0 + 4 * g4 + i16;
            *dst = (k0 == klast ? 0.f : *dst) + pick4(Rp, i16);
          }
        }
      }
    }
    __syncthreads();

    // ---- token values R_t, A_t and key norms ----
    if (tid < n) {
      const int t = tid;
      float s = 0.f, am = 0.f;
#pragma unroll
      for (int w2 = 0; w2 < RWV; ++w2)
        if (16 * w2 < dm.W) { s += sRp[w2 * NMAX + t]; am += sAp[w2 * NMAX + t]; }
      float R = s / Sg;
      if (tv.dhat) R = (1.f - dm.lam_graph) * R + dm.lam_graph * tv.dhat[a0 + t];   // eq:app_bottom_up_value
      const float A = am / (float)dm.W;
      sR[t] = R;
      sA[t] = A;
      tv.tok_R[(int64_t)lg * dm.N_c + a0 + t] = R;
      tv.tok_A[(int64_t)lg * dm.N_c + a0 + t] = A;
    }
    __syncthreads();

    // ---- per-dimension sums of R v and v over the unit ----
    {
      const int d = tid % D, q2 = tid / D;
      float sv = 0.f, srv = 0.f;
      for (int t = q2; t < n; t += Lay::NPV) {
        const float v = ldf(sVt, d * Lay::LDV + t);
        sv += v;
        srv += sR[t] * v;
      }
      sPv[q2 * D + d] = srv;
      sPs[q2 * D + d] = sv;
    }
    __syncthreads();

    // ---- root prototype (wave 0) ----
    if (w == 0) {
      float sr = 0.f, sa = 0.f, skn = 0.f;
      for (int t = lane; t < n; t += 64) { sr += sR[t]; sa += sA[t]; skn += sKn[t]; }
      sr = wave_sum(sr);
      sa = wave_sum(sa);
      skn = wave_sum(skn);
      const float inv = 1.0f / (float)n;
      constexpr int DL = D / 64;              // dims per lane: lane + 64 h
      float kb[DL];
      float ss = 0.f;
#pragma unroll
      for (int h = 0; h < DL; ++h) {
        const int d = lane + 64 * h;
        float s = 0.f;
#pragma unroll
        for (int q = 0; q < Lay::NPK; ++q) s += sPk[q * D + d];
        kb[h] = s * inv;
        ss += kb[h] * kb[h];
      }
      ss = wave_sum(ss);
      const float coh = sqrtf(ss) / (skn * inv + dm.eps);
      const float me = fminf(fmaxf((float)n * coh * coh, 1.0f), (float)n);
      if constexpr (D == 128) {               // lane holds the pair (lane, lane + 64)
        sKt[lane] = kb[0] * pcos - kb[1] * psin;
        sKt[lane + H2] = kb[1] * pcos + kb[0] * psin;
      } else {                                // D == 64: partner dim lane ^ 32
        const float other = __shfl_xor(kb[0], 32, 64);
        sKt[lane] = lane < 32 ? kb[0] * pcos - other * psin : kb[0] * pcos + other * psin;
      }
      const float beta = dm.beta_frac * sr * inv;
      const float den = sr + (float)n * beta + dm.eps;
#pragma unroll
      for (int h = 0; h < DL; ++h) {
        const int d = lane + 64 * h;
        float vr = 0.f, vs = 0.f;
#pragma unroll
        for (int q = 0; q < Lay::NPV; ++q) { vr += sPv[q * D + d]; vs += sPs[q * D + d]; }
        sVv[d] = (vr + beta * vs) / den;
      }
      if (lane == 0) { sRed[0] = sr; sRed[1] = sa; sRed[2] = me; }
    }
    __syncthreads();
    if (tid < 2 * D) {                        // the unit's root prototype, as pack writes it
      T* pr = (T*)tv.proto + unit * 2 * D;
      stf(pr, tid, tid < D ? sKt[tid] : sVv[tid - D]);
    }
    if (tid == 0) tv.proto_logm[unit] = logf(sRed[2]);

    // ---- distortion of the root: probes of wave w (head slot 0 is in qr[0]) ----
    {
      float con = 0.f;
      if (wave_on) {
        const float me = sRed[2];
        float qk = 0.f;
#pragma unroll
        for (int e = 0; e < QE; ++e) {
          float qv;
          if constexpr (BF) qv = __uint_as_float(e & 1 ? (qr[0][e >> 1] & 0xffff0000u) : (qr[0][e >> 1] << 16));
          else qv = __uint_as_float(qr[0][e]);
          qk += qv * sKt[QE * g4 + e];
        }
        qk += __shfl_xor(qk, 16, 64);
        qk += __shfl_xor(qk, 32, 64);
        const float z = me * fexp(qk * scale - mq);
        float Z = Zl;
        Z += __shfl_xor(Z, 16, 64);
        Z += __shfl_xor(Z, 32, 64);
        float s1 = 0.f, s2 = 0.f;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const float4 vv = *(const float4*)(sVv + 16 * dt + 4 * g4);
          const float vt[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float M = Macc[dt][r];
            const float df = M - z * vt[r];
            s1 += df * df;
            s2 += M * M;
          }
        }
        s1 += __shfl_xor(s1, 16, 64);
        s1 += __shfl_xor(s1, 32, 64);
        s2 += __shfl_xor(s2, 16, 64);
        s2 += __shfl_xor(s2, 32, 64);
        const float dz = Z - z;
        const float Dq = dm.lam_Z * dz * dz / (Z * Z + dm.eps) + dm.lam_M * s1 / (s2 + dm.eps);
        con = (uok && g4 == 0) ? (Z * zcq) * Dq : 0.f;
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) con += __shfl_xor(con, o, 64);
      }
      if (lane == 0) sRed[4 + w] = con;
    }
    __syncthreads();

    // ---- outputs: root node, Add key, empty Split slots ----
    if (tid == 0) {
      const float sr = sRed[0], dd = sRed[1];
      float Dv = 0.f;
      for (int w2 = 0; w2 < RWV; ++w2) Dv += sRed[4 + w2];
      Dv = n >= 2 ? Dv / (float)dm.W : 0.f;
      const int64_t sl = (int64_t)lg * 2 * dm.N_c + 2 * a0;
      tv.node_a[sl] = (int32_t)a0;
      tv.node_n[sl] = n;
      tv.node_child[sl] = -1;
      tv.node_parent[sl] = -1;
      tv.node_nch[sl] = 0;
      tv.node_kind[sl] = 0;
      tv.node_cut[sl] = -1;
      tv.node_D[sl] = Dv;
      tv.node_R[sl] = sr;
      tv.unit_nn[unit] = 1;
      tv.unit_Ddrop[unit] = dd;
      const uint32_t ord = (uint32_t)lg * (uint32_t)J + (uint32_t)j;
      const float Ua = utility(add_gain(om, sr, dd, Dv), 1);
      tv.add_U[unit] = Ua;
      tv.add_E[unit] = op_key(Ua, ord * 256u);
      tv.add_exec[unit] = 0;
    }
    for (int i = tid; i < 2 * n; i += RT) {
      const int64_t sl = (int64_t)lg * 2 * dm.N_c + 2 * a0 + i;
      tv.sp_U[sl] = 0.f;
      tv.sp_E[sl] = 0;
      tv.sp_cost[sl] = 0;
      tv.sp_exec[sl] = 0;
    }
  }
}

hipError_t launch_root(const Dims& dm, const void* K, const void* V, const void* Q, const float* cosT,
                       const float* sinT, const int32_t* slot_starts, const int32_t* n_slots, const TreeView& tv,
                       hipStream_t st) {
  const int64_t cap = (int64_t)dm.L * dm.G * dm.J_cap;
  const dim3 grid((unsigned)(cap < ROOT_GRID ? cap : ROOT_GRID));
  const int lds = root_lds_bytes(dm);
#define GKV_LAUNCH_ROOT(TT, DD)                                                                            \
  do {                                                                                                     \
    auto fn = dm.hpg > 4 ? k_root<TT, DD, true> : k_root<TT, DD, false>;                                   \
    hipError_t e0 = hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds); \
    if (e0 != hipSuccess) return e0;                                                                       \
    hipLaunchKernelGGL(fn, grid, dim3(RT), lds, st, dm, (const TT*)K, (const TT*)V, (const TT*)Q, cosT, sinT, \
                       slot_starts, n_slots, tv);                                                          \
  } while (0)
  if (dm.dtype == GRACEKV_BF16) {
    return launch_root_bf16(dm, K, V, Q, cosT, sinT, slot_starts, n_slots, tv, st);
  } else {
    if (dm.d != 64) return hipErrorInvalidValue;   // fp32 caches take d = 64 only
    GKV_LAUNCH_ROOT(float, 64);
  }
#undef GKV_LAUNCH_ROOT
  return hipGetLastError();
}

}  // namespace gkv
