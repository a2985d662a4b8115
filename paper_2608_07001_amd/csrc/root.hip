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
// up to 2 heads are held in registers at a time.
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
  static constexpr int NPK = RT / (D / 2);              // token phases of the k° sums
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
  constexpr int HG = BF ? 2 : 1;             // heads per register group
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
  const int ngr = (dm.hpg + HG - 1) / HG;

  uint32_t qreg[HG][QW];                      // Q quarter rows (head slots k0 .. k0+HG-1)
  float2 rs[HG];                              // (m_V, Z_V) of the lane's rows
  float mq = 0.f, zcq = 1.f;                  // probe shift and Z_q(C)

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
    // Q quarter rows and row statistics of head group gr (issued early for the last group)
    auto load_q = [&](int gr) {
      const int k0 = gr * HG;
#pragma unroll
      for (int kk = 0; kk < HG; ++kk) {
        if (k0 + kk < dm.hpg) {
          const int hl = (hp + k0 + kk) % dm.hpg;
          const uint4* q4 = (const uint4*)(Q + (((int64_t)l * dm.H + (int64_t)g * dm.hpg + hl) * dm.W + uq) * D + QE * g4);
#pragma unroll
          for (int h = 0; h < QW / 4; ++h) {
            const uint4 v = q4[h];
            qreg[kk][4 * h] = v.x; qreg[kk][4 * h + 1] = v.y; qreg[kk][4 * h + 2] = v.z; qreg[kk][4 * h + 3] = v.w;
          }
          const float4 st = tv.row_stats[(int64_t)lg * dm.rows + hl * dm.W + uq];
          rs[kk] = make_float2(st.x, st.y);
        }
      }
    };
    if (wave_on) {
      load_q(ngr - 1);
      mq = tv.probe_m[(int64_t)lg * dm.W + uq];
      zcq = tv.probe_ZC[(int64_t)lg * dm.W + uq];
    }
    __syncthreads();                          // the previous unit is done with LDS

    // ---- stage K (row-major) and V (transposed), zero past n ----
    if constexpr (BF) {
      constexpr int CPR = D / 8;              // 16-byte chunks per row
      // lane -> (token pair, chunk): 8 pairs x CPR chunks per group
      for (int e = tid; e < (rows16 / 2) * CPR; e += RT) {
        const int grp = e / (8 * CPR), rem = e % (8 * CPR);
        const int c = rem / 8, t = 2 * (8 * grp + rem % 8);
        uint4 k0 = make_uint4(0, 0, 0, 0), k1 = k0, v0 = k0, v1 = k0;
        if (t < n) { k0 = *(const uint4*)(Kp + (int64_t)t * D + 8 * c); v0 = *(const uint4*)(Vp + (int64_t)t * D + 8 * c); }
        if (t + 1 < n) { k1 = *(const uint4*)(Kp + (int64_t)(t + 1) * D + 8 * c); v1 = *(const uint4*)(Vp + (int64_t)(t + 1) * D + 8 * c); }
        *(uint4*)(sK + t * Lay::LDK + 8 * c) = k0;
        *(uint4*)(sK + (t + 1) * Lay::LDK + 8 * c) = k1;
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
        float4 kk = make_float4(0.f, 0.f, 0.f, 0.f), vv = kk;
        if (t < n) { kk = *(const float4*)(Kp + (int64_t)t * D + 4 * c); vv = *(const float4*)(Vp + (int64_t)t * D + 4 * c); }
        *(float4*)(sK + t * Lay::LDK + 4 * c) = kk;
        sVt[(4 * c + 0) * Lay::LDV + t] = vv.x;
        sVt[(4 * c + 1) * Lay::LDV + t] = vv.y;
        sVt[(4 * c + 2) * Lay::LDV + t] = vv.z;
        sVt[(4 * c + 3) * Lay::LDV + t] = vv.w;
      }
    }
    for (int e = tid; e < RWV * NMAX; e += RT) { sRp[e] = 0.f; sAp[e] = 0.f; }
    __syncthreads();

    // ---- logits, relevance, probe exponentials and M^T = V^T E^T ----
    f32x4 Macc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) Macc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float Zl = 0.f;
    if (wave_on) {
      // head groups in reverse so that the probe head (slot 0) is in registers at the end
      for (int gr = ngr - 1; gr >= 0; --gr) {
        const int k0 = gr * HG;
        if (gr != ngr - 1) load_q(gr);
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
          float Rp[4] = {0.f, 0.f, 0.f, 0.f}, ev[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kk = 0; kk < HG; ++kk) {
            if (k0 + kk < dm.hpg) {
              f32x4 acc = {0.f, 0.f, 0.f, 0.f};
              if constexpr (BF) {
#pragma unroll
                for (int s = 0; s < QE / 4; ++s)
                  acc = mfma_bf16_16x16x16(pk4(kreg[2 * s], kreg[2 * s + 1]),
                                           pk4(qreg[kk][2 * s], qreg[kk][2 * s + 1]), acc);
              } else {
#pragma unroll
                for (int s = 0; s < QE; ++s)
                  acc = mfma_f32_16x16x4(__uint_as_float(kreg[s]), __uint_as_float(qreg[kk][s]), acc);
              }
              // lane holds tokens t0 + 4 g4 + r of the lane's query row
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                if (uok && t0 + 4 * g4 + r < n) {
                  const float x = acc[r] * scale;
                  Rp[r] += expf(x - rs[kk].x) / rs[kk].y;
                  if (gr == 0 && kk == 0) ev[r] = expf(x - mq);
                }
              }
            }
          }
          if (gr == 0) {
            float ap[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) { ap[r] = ev[r] / zcq; Zl += ev[r]; }
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
            for (int o = 1; o < 16; o <<= 1)
#pragma unroll
              for (int r = 0; r < 4; ++r) ap[r] += __shfl_xor(ap[r], o, 64);
            if (i16 < 4) sAp[w * NMAX + t0 + 4 * g4 + i16] = pick4(ap, i16);
          }
#pragma unroll
          for (int o = 1; o < 16; o <<= 1)
#pragma unroll
            for (int r = 0; r < 4; ++r) Rp[r] += __shfl_xor(Rp[r], o, 64);
          if (i16 < 4) sRp[w * NMAX + t0 + 4 * g4 + i16] += pick4(Rp, i16);
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
      float kn = 0.f;
      for (int c = 0; c < D; ++c) {
        const float x = ldf(sK, t * Lay::LDK + c);
        kn += x * x;
      }
      sKn[t] = sqrtf(kn);
    }
    __syncthreads();

    // ---- per-dimension sums over the unit: k° (RoPE undone at t), R v and v ----
    {
      const int i = tid % H2, q = tid / H2;
      float s0 = 0.f, s1 = 0.f;
      for (int tb = q; tb < n; tb += 4 * Lay::NPK) {
        float c8[4], s8[4], a8[4], b8[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int t = tb + v * Lay::NPK;
          const int tt = t < n ? t : n - 1;
          const int64_t ta = a0 + tt;
          c8[v] = cosT[ta * H2 + i];
          s8[v] = sinT[ta * H2 + i];
          a8[v] = ldf(sK, tt * Lay::LDK + i);
          b8[v] = ldf(sK, tt * Lay::LDK + i + H2);
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          if (tb + v * Lay::NPK < n) {
            s0 += a8[v] * c8[v] + b8[v] * s8[v];
            s1 += b8[v] * c8[v] - a8[v] * s8[v];
          }
        }
      }
      sPk[q * D + i] = s0;
      sPk[q * D + i + H2] = s1;
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
      const int64_t p = round_half_even_mid((int)a0, (int)a0 + n);
      if constexpr (D == 128) {               // lane holds the pair (lane, lane + 64)
        const float c = cosT[p * H2 + lane], sn = sinT[p * H2 + lane];
        sKt[lane] = kb[0] * c - kb[1] * sn;
        sKt[lane + H2] = kb[1] * c + kb[0] * sn;
      } else {                                // D == 64: partner dim lane ^ 32
        const float other = __shfl_xor(kb[0], 32, 64);
        const int i = lane & 31;
        const float c = cosT[p * H2 + i], sn = sinT[p * H2 + i];
        sKt[lane] = lane < 32 ? kb[0] * c - other * sn : kb[0] * c + other * sn;
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
          if constexpr (BF) qv = __uint_as_float(e & 1 ? (qreg[0][e >> 1] & 0xffff0000u) : (qreg[0][e >> 1] << 16));
          else qv = __uint_as_float(qreg[0][e]);
          qk += qv * sKt[QE * g4 + e];
        }
        qk += __shfl_xor(qk, 16, 64);
        qk += __shfl_xor(qk, 32, 64);
        const float z = me * expf(qk * scale - mq);
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
        con = (uok && g4 == 0) ? (Z / zcq) * Dq : 0.f;
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
