// Root evaluation of every (layer, KV head, slot) unit.
//
// For each unit [a0, a0 + n) of one (l, g) this computes, in one pass over the
// unit's keys and values:
//   * pass 2 of the direct relevance (App. A.4 eq:app_attention_probability,
//     eq:app_direct_relevance, lambda_graph = 0 so R^tok = s-hat): R_t for each
//     token, from the row statistics of pass 1;
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
  static constexpr int oK = 0;
  static constexpr int oVt = oK + NMAX * LDK * (int)sizeof(T);
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
  static constexpr int bytes = oRed + 16 * 4;
};

int root_lds_bytes(const Dims& dm) {
  if (dm.dtype == GRACEKV_BF16) return dm.d == 128 ? RootLds<uint16_t, 128>::bytes : RootLds<uint16_t, 64>::bytes;
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

template <typename T, int D>
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

  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, i16 = lane & 15, g4 = lane >> 4;
  const int J = *n_slots;
  if (J < 1 || J > dm.J_cap) {                // malformed partition: nothing to build
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(tv.status, 2);
    return;
  }
  const int64_t total = (int64_t)dm.L * dm.G * J;
  const int64_t per = (total + gridDim.x - 1) / gridDim.x;
  const int64_t ub = (int64_t)blockIdx.x * per;
  const int64_t ue = ub + per < total ? ub + per : total;
  const float scale = 1.0f / sqrtf((float)D);
  const int u = 16 * w + i16;                 // the lane's window query
  const bool uok = u < dm.W;
  const int uq = uok ? u : 0;
  const int hp = uq % dm.hpg;                 // query head of probe u
  const bool wave_on = 16 * w < dm.W;

  constexpr int CHP = H2 / 8;                // 8-dim pair chunks per token in the k° staging
  uint32_t qa[QW], qb[QW];                    // Q quarter rows: current head, next head
  float2 rsa = make_float2(0.f, 1.f), rsb = rsa;   // (m_V, 1 / Z_V) of the lane's rows
  float mq = 0.f, zcq = 1.f;                  // probe shift and 1 / Z_q(C)

  for (int64_t uu = ub; uu < ue; ++uu) {
    const int lg = (int)(uu / J), j = (int)(uu % J);
    const int l = lg / dm.G, g = lg % dm.G;
    const int64_t unit = (int64_t)lg * dm.J_cap + j;
    const int64_t a0 = slot_starts[j];
    const int n = slot_starts[j + 1] - (int)a0;
    if (n < 1 || n > NMAX || a0 < 0 || a0 + n > dm.N_c) {   // malformed partition: refuse the unit
      if (tid == 0) { atomicOr(tv.status, 2); tv.unit_nn[unit] = 0; }
      continue;
    }
    const int rows16 = (n + 15) & ~15;
    const int n_tt = rows16 / 16;
    const T* Kp = K + ((int64_t)lg * dm.T + a0) * D;
    const T* Vp = V + ((int64_t)lg * dm.T + a0) * D;
    // Q quarter row and row statistics of head slot k (head (hp + k) mod |H(g)|)
    auto load_q = [&](int k, uint32_t* q, float2& rsv) {
      const int hl = (hp + k) % dm.hpg;
      const uint4* q4 = (const uint4*)(Q + (((int64_t)l * dm.H + (int64_t)g * dm.hpg + hl) * dm.W + uq) * D + QE * g4);
#pragma unroll
      for (int h = 0; h < QW / 4; ++h) {
        const uint4 v = q4[h];
        q[4 * h] = v.x; q[4 * h + 1] = v.y; q[4 * h + 2] = v.z; q[4 * h + 3] = v.w;
      }
      const float4 st = tv.row_stats[(int64_t)lg * dm.rows + hl * dm.W + uq];
      rsv = make_float2(st.x, 1.0f / st.y);      // (m_V, 1 / Z_V)
    };
    if (wave_on) {
      load_q(dm.hpg - 1, qa, rsa);
      mq = tv.probe_m[(int64_t)lg * dm.W + uq];
      zcq = 1.0f / tv.probe_ZC[(int64_t)lg * dm.W + uq];
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
      for (int e = tid; e < rows16 * CHP; e += RT) {
        const int t = e / CHP;
        float k1[8], k2[8], o1[8], o2[8];
        if constexpr (BF) {
          uint4 u1 = make_uint4(0, 0, 0, 0), u2 = u1;
          if (t < n) { u1 = *(const uint4*)(Kp + (int64_t)t * D + c); u2 = *(const uint4*)(Kp + (int64_t)t * D + c + H2); }
          *(uint4*)(sK + t * Lay::LDK + c) = u1;
          *(uint4*)(sK + t * Lay::LDK + c + H2) = u2;
          const uint32_t w1[4] = {u1.x, u1.y, u1.z, u1.w}, w2[4] = {u2.x, u2.y, u2.z, u2.w};
#pragma unroll
          for (int h = 0; h < 4; ++h) {
            k1[2 * h] = __uint_as_float(w1[h] << 16); k1[2 * h + 1] = __uint_as_float(w1[h] & 0xffff0000u);
            k2[2 * h] = __uint_as_float(w2[h] << 16); k2[2 * h + 1] = __uint_as_float(w2[h] & 0xffff0000u);
          }
        } else {
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
        }
        float ss = 0.f;
        if (t < n) {
          const int64_t ta = a0 + t;
          const float4 c0 = *(const float4*)(cosT + ta * H2 + c), c1 = *(const float4*)(cosT + ta * H2 + c + 4);
          const float4 s0 = *(const float4*)(sinT + ta * H2 + c), s1 = *(const float4*)(sinT + ta * H2 + c + 4);
          const float cs8[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
          const float sn8[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
#pragma unroll
          for (int h = 0; h < 8; ++h) {
            o1[h] = k1[h] * cs8[h] + k2[h] * sn8[h];
            o2[h] = k2[h] * cs8[h] - k1[h] * sn8[h];
            kacc[h] += o1[h];
            kacc[8 + h] += o2[h];
            ss += o1[h] * o1[h] + o2[h] * o2[h];
          }
        }
#pragma unroll
        for (int o = 1; o < CHP; o <<= 1) ss += __shfl_xor(ss, o, 64);
        if (t < n && c == 0) sKn[t] = sqrtf(ss);
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
    if constexpr (BF) {
      constexpr int CPR = D / 8;              // 16-byte chunks per row
      // lane -> (token pair, chunk): 8 pairs x CPR chunks per group
      for (int e = tid; e < (rows16 / 2) * CPR; e += RT) {
        const int grp = e / (8 * CPR), rem = e % (8 * CPR);
        const int c = rem / 8, t = 2 * (8 * grp + rem % 8);
        uint4 v0 = make_uint4(0, 0, 0, 0), v1 = v0;
        if (t < n) v0 = *(const uint4*)(Vp + (int64_t)t * D + 8 * c);
        if (t + 1 < n) v1 = *(const uint4*)(Vp + (int64_t)(t + 1) * D + 8 * c);
        const uint32_t a[4] = {v0.x, v0.y, v0.z, v0.w}, b[4] = {v1.x, v1.y, v1.z, v1.w};
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          *(uint32_t*)(sVt + (8 * c + 2 * h) * Lay::LDV + t) = (a[h] & 0xffffu) | (b[h] << 16);
          *(uint32_t*)(sVt + (8 * c + 2 * h + 1) * Lay::LDV + t) = (a[h] >> 16) | (b[h] & 0xffff0000u);
        }
      }
    } else {
      constexpr int CPR = D / 4;
      for (int e = tid; e < rows16 * CPR; e += RT) {
        const int grp = e / (16 * CPR), rem = e % (16 * CPR);
        const int c = rem / 16, t = 16 * grp + rem % 16;
        float4 vv = make_float4(0.f, 0.f, 0.f, 0.f);
        if (t < n) vv = *(const float4*)(Vp + (int64_t)t * D + 4 * c);
        sVt[(4 * c + 0) * Lay::LDV + t] = vv.x;
        sVt[(4 * c + 1) * Lay::LDV + t] = vv.y;
        sVt[(4 * c + 2) * Lay::LDV + t] = vv.z;
        sVt[(4 * c + 3) * Lay::LDV + t] = vv.w;
      }
    }
    for (int e = tid; e < RWV * NMAX; e += RT) { sRp[e] = 0.f; sAp[e] = 0.f; }
    __syncthreads();

    // ---- logits, relevance, probe exponentials and M^T = V^T E^T: heads one
    // at a time with the next head's Q in flight, the probe head (slot 0) last ----
    f32x4 Macc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) Macc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float Zl = 0.f;
    if (wave_on) {
      for (int k = dm.hpg - 1; k >= 0; --k) {
        if (k > 0) load_q(k - 1, qb, rsb);
        for (int tb = 0; tb < n_tt; ++tb) {
          const int t0 = 16 * tb;
          uint32_t kreg[QW];
          {
            const uint4* k4 = (const uint4*)(sK + (t0 + i16) * Lay::LDK + QE * g4);
#pragma unroll
            for (int h = 0; h < QW / 4; ++h) {
              const uint4 v = k4[h];
              kreg[4 * h] = v.x; kreg[4 * h + 1] = v.y; kreg[4 * h + 2] = v.z; kreg[4 * h + 3] = v.w;
            }
          }
          f32x4 acc = {0.f, 0.f, 0.f, 0.f};
          if constexpr (BF) {
#pragma unroll
            for (int s = 0; s < QE / 4; ++s)
              acc = mfma_bf16_16x16x16(pk4(kreg[2 * s], kreg[2 * s + 1]), pk4(qa[2 * s], qa[2 * s + 1]), acc);
          } else {
#pragma unroll
            for (int s = 0; s < QE; ++s)
              acc = mfma_f32_16x16x4(__uint_as_float(kreg[s]), __uint_as_float(qa[s]), acc);
          }
          // lane holds tokens t0 + 4 g4 + r of the lane's query row
          float Rp[4], ev[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            Rp[r] = 0.f;
            if (uok && t0 + 4 * g4 + r < n) {
              const float x = acc[r] * scale;
              Rp[r] = fexp(x - rsa.x) * rsa.y;
              if (k == 0) ev[r] = fexp(x - mq);
            }
          }
          if (k == 0) {
            float ap[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) { ap[r] = ev[r] * zcq; Zl += ev[r]; }
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
          if (i16 < 4) sRp[w * NMAX + t0 + 4 * g4 + i16] += pick4(Rp, i16);
        }
        if (k > 0) {
#pragma unroll
          for (int h = 0; h < QW; ++h) qa[h] = qb[h];
          rsa = rsb;
        }
      }
    }
    __syncthreads();

    // ---- token values R_t, A_t and key norms ----
    if (tid < n) {
      const int t = tid;
      float s = 0.f, am = 0.f;
#pragma unroll
      for (int w2 = 0; w2 < RWV; ++w2) { s += sRp[w2 * NMAX + t]; am += sAp[w2 * NMAX + t]; }
      const float R = s / (tv.lg_S[lg] + dm.eps);
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

    // ---- distortion of the root: probes of wave w ----
    {
      float con = 0.f;
      if (wave_on) {
        const float me = sRed[2];
        float qk = 0.f;
#pragma unroll
        for (int e = 0; e < QE; ++e) {
          float qv;
          if constexpr (BF) qv = __uint_as_float(e & 1 ? (qa[e >> 1] & 0xffff0000u) : (qa[e >> 1] << 16));
          else qv = __uint_as_float(qa[e]);
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
      const float Ua = utility(add_gain(tv.omega[lg], sr, dd, Dv), 1);
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
    auto fn = k_root<TT, DD>;                                                                              \
    hipError_t e0 = hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds); \
    if (e0 != hipSuccess) return e0;                                                                       \
    hipLaunchKernelGGL(fn, grid, dim3(RT), lds, st, dm, (const TT*)K, (const TT*)V, (const TT*)Q, cosT, sinT, \
                       slot_starts, n_slots, tv);                                                          \
  } while (0)
  if (dm.dtype == GRACEKV_BF16) {
    if (dm.d == 128) GKV_LAUNCH_ROOT(uint16_t, 128); else GKV_LAUNCH_ROOT(uint16_t, 64);
  } else {
    if (dm.d == 128) GKV_LAUNCH_ROOT(float, 128); else GKV_LAUNCH_ROOT(float, 64);
  }
#undef GKV_LAUNCH_ROOT
  return hipGetLastError();
}

}  // namespace gkv
