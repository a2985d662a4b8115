// Prototype-tree refinement, one workgroup per (layer, KV head, slot) unit.
//
// Implements App. A.3 (RoPE-consistent key prototype eq:app_rope_prototype,
// value prototype eq:app_value_prototype, effective multiplicity
// eq:app_effective_multiplicity, distortion eq:app_original_attention_stats ..
// eq:app_node_and_drop_distortion, recursive refinement eq:app_binary_split ..
// eq:app_split_choice).  The root of every unit, the token values R_t and the
// probe masses A_t come from the root kernel; this kernel resumes from the node
// table.
//
// Per unit (n <= 128 tokens), 512 threads:
//   1. K and V tiles go to LDS; the matrix cores form the logits of the W
//      distortion probes against the unit's keys, giving
//      e_{q,t} = exp(l_{q,t} - m_q) (kept in LDS, fp32).
//   2. The tree is refined top-down in BFS order.  For node [a, b) the binary
//      cuts (top-16 curvature positions t -> cut t+1, plus the midpoint) and the
//      extraction token p define children that are all prefixes [a, x) or
//      suffixes [x, b) of the node.  The two halves of the workgroup sweep the
//      node at the same time, one left to right (prefix children) and one right
//      to left (suffix children): running sums of k°, R v, v, R and ||k||, and per
//      probe of e and e v, are read off at each cut, so a child costs O(W d)
//      once its sweep has passed it.  Loads are issued 8 (prototype sums) or 4
//      (probe sums) tokens ahead.
//   3. Scores are compared in fp32 (binary form wins ties, smaller cut wins
//      ties), children are appended, and the node table is written out.
#include "common.h"

namespace gkv {

constexpr int BT = 512;          // threads per unit
constexpr int GT = 256;          // threads per sweep group
constexpr int TPQ = 4;           // threads per probe in the probe sweep
constexpr int CM = 18;           // children per sweep: up to 17 cuts + one extraction side
constexpr int ES = NMAX + 1;     // row stride of the probe exponentials (odd: no bank conflicts across probes)

template <typename T> struct BPad;
template <> struct BPad<uint16_t> { static constexpr int v = 4; };
template <> struct BPad<float> { static constexpr int v = 1; };

template <typename T, int D>
struct BuildLds {
  static constexpr int LDK = D + BPad<T>::v;
  static constexpr int oK = 0;
  static constexpr int oV = oK + NMAX * LDK * (int)sizeof(T);
  static constexpr int oE = ((oV + NMAX * D * (int)sizeof(T)) + 15) & ~15;
  static constexpr int oR = oE + WMAX * ES * 4;
  static constexpr int oKap = oR + NMAX * 4;
  static constexpr int oA = oKap + NMAX * 4;
  static constexpr int oKn = oA + NMAX * 4;
  static constexpr int oNa = oKn + NMAX * 4;
  static constexpr int oNn = oNa + 256 * 4;
  static constexpr int oNc = oNn + 256 * 4;
  static constexpr int oNp = oNc + 256 * 4;
  static constexpr int oNch = oNp + 256 * 4;
  static constexpr int oNk = oNch + 256 * 4;
  static constexpr int oNcut = oNk + 256 * 4;
  static constexpr int oND = oNcut + 256 * 4;
  static constexpr int oNR = oND + 256 * 4;
  // per sweep group g: child mean k° / k~ [CM][D], child v~ [CM][D], contributions [CM][WMAX]
  static constexpr int oCk = oNR + 256 * 4;
  static constexpr int oCv = oCk + 2 * CM * D * 4;
  static constexpr int oCon = oCv + 2 * CM * D * 4;
  static constexpr int oCs = oCon + 2 * CM * WMAX * 4;       // child scalars [2][8][CM]
  static constexpr int oX = oCs + 2 * 8 * CM * 4;            // cut lists and misc ints
  static constexpr int oFlag = oX + 4 * 64 * 4;
  static constexpr int oNE = oFlag + NMAX * 4;                // effective key of each node's creating op
  static constexpr int oNU = oNE + 256 * 8;                   // utility of each node's Split
  static constexpr int bytes = oNU + 256 * 4;
};

int build_lds_bytes(const Dims& dm) {
  if (dm.dtype == GRACEKV_BF16) return dm.d == 128 ? BuildLds<uint16_t, 128>::bytes : BuildLds<uint16_t, 64>::bytes;
  return dm.d == 128 ? BuildLds<float, 128>::bytes : BuildLds<float, 64>::bytes;
}

// child scalar rows in cs: 0 n, 1 sumR, 2 mean||k||, 3 m_eff, 4 p, 5 D
template <typename T, int D>
struct Unit {
  using Lay = BuildLds<T, D>;
  char* s;
  T* sK; T* sV; float* sE; float* sR; float* sKap; float* sA; float* sKn;
  int* na; int* nn; int* nc; int* np; int* nch; int* nk; int* ncut; float* nD; float* nR;
  float* ck; float* cv; float* con; float* cs; int* xi; int* flag;
  uint64_t* nE; float* nU;
  __device__ Unit(char* base) : s(base) {
    sK = (T*)(s + Lay::oK); sV = (T*)(s + Lay::oV); sE = (float*)(s + Lay::oE); sR = (float*)(s + Lay::oR);
    sKap = (float*)(s + Lay::oKap); sA = (float*)(s + Lay::oA); sKn = (float*)(s + Lay::oKn);
    na = (int*)(s + Lay::oNa); nn = (int*)(s + Lay::oNn); nc = (int*)(s + Lay::oNc); np = (int*)(s + Lay::oNp);
    nch = (int*)(s + Lay::oNch); nk = (int*)(s + Lay::oNk); ncut = (int*)(s + Lay::oNcut);
    nD = (float*)(s + Lay::oND); nR = (float*)(s + Lay::oNR);
    ck = (float*)(s + Lay::oCk); cv = (float*)(s + Lay::oCv); con = (float*)(s + Lay::oCon);
    cs = (float*)(s + Lay::oCs); xi = (int*)(s + Lay::oX); flag = (int*)(s + Lay::oFlag);
    nE = (uint64_t*)(s + Lay::oNE); nU = (float*)(s + Lay::oNU);
  }
  __device__ float* gck(int g) { return ck + g * CM * D; }
  __device__ float* gcv(int g) { return cv + g * CM * D; }
  __device__ float* gcon(int g) { return con + g * CM * WMAX; }
  __device__ float* gcs(int g, int row) { return cs + (g * 8 + row) * CM; }
};

// DPT consecutive elements of an LDS row as fp32 (16-byte aligned chunks)
template <int DPT>
__device__ __forceinline__ void lds_row(const uint16_t* p, float* out) {
  const uint4* q = (const uint4*)p;
#pragma unroll
  for (int k = 0; k < DPT / 8; ++k) {
    const uint4 w = q[k];
    const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      out[8 * k + 2 * h] = __uint_as_float(ws[h] << 16);
      out[8 * k + 2 * h + 1] = __uint_as_float(ws[h] & 0xffff0000u);
    }
  }
}
template <int DPT>
__device__ __forceinline__ void lds_row(const float* p, float* out) {
  const float4* q = (const float4*)p;
#pragma unroll
  for (int k = 0; k < DPT / 4; ++k) {
    const float4 w = q[k];
    out[4 * k] = w.x; out[4 * k + 1] = w.y; out[4 * k + 2] = w.z; out[4 * k + 3] = w.w;
  }
}

// Both sweeps of one node at once.  Group 0 evaluates the prefix children
// [a, XL[c]), group 1 the suffix children [XR[c], b) (0-based inside the unit,
// absolute start a0).  Per child: rows 0 n, 1 sum R, 5 D of the group's cs.
template <typename T, int D>
__device__ void sweep2(Unit<T, D>& U, const Dims& dm, int a, int b, const int* XL, int nl, const int* XR, int nr,
                       int64_t a0, const float* __restrict__ cosT, const float* __restrict__ sinT, const float* qv,
                       float m_q, float zc_q, float scale) {
  using Lay = BuildLds<T, D>;
  constexpr int H2 = D / 2;
  constexpr int DPT = D / TPQ;
  const int tid = threadIdx.x;
  const int g = tid / GT, lt = tid % GT;
  const bool prefix = g == 0;
  const int* xs = prefix ? XL : XR;
  const int nx = prefix ? nl : nr;
  float* ck = U.gck(g);
  float* cv = U.gcv(g);
  float* con = U.gcon(g);
  float* cn = U.gcs(g, 0);
  float* cR = U.gcs(g, 1);
  float* cKm = U.gcs(g, 2);
  float* cMe = U.gcs(g, 3);
  float* cD = U.gcs(g, 5);
  const int t_first = prefix ? a : b - 1;
  const int step = prefix ? 1 : -1;
  const int t_last = nx > 0 ? (prefix ? xs[nx - 1] - 1 : xs[0]) : t_first;
  const int steps = nx > 0 ? (prefix ? t_last - t_first + 1 : t_first - t_last + 1) : 0;
  // ---- phase A: prototype sums, loads 8 tokens ahead.  Threads lt < D sum
  // k° of dimension lt (and the scalars); threads D <= lt < 2D sum R v and v of
  // dimension lt - D. ----
  if (lt < 2 * D && steps > 0) {
    const bool kside = lt < D;
    const int i = kside ? lt : lt - D;
    const int ih = i < H2 ? i : i - H2;
    const int ip = i < H2 ? i + H2 : i - H2;
    float s0 = 0.f, s1 = 0.f, sr = 0.f, skn = 0.f;
    int ci = prefix ? 0 : nx - 1;
    int xnext = xs[ci];
    bool done = false;
    for (int it0 = 0; it0 < steps && !done; it0 += 8) {
      float f0[8], f1[8], f2[8], f3[8], r8[8], k8[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int it = min(it0 + u, steps - 1);
        const int t = t_first + step * it;
        if (kside) {
          const int64_t ta = a0 + t;
          f0[u] = cosT[ta * H2 + ih];
          f1[u] = sinT[ta * H2 + ih];
          f2[u] = ldf(U.sK, t * Lay::LDK + i);
          f3[u] = ldf(U.sK, t * Lay::LDK + ip);
          k8[u] = U.sKn[t];
        } else {
          f0[u] = ldf(U.sV, t * D + i);
        }
        r8[u] = U.sR[t];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (done || it0 + u >= steps) break;
        const int t = t_first + step * (it0 + u);
        if (kside) {
          s0 += i < H2 ? f2[u] * f0[u] + f3[u] * f1[u] : f2[u] * f0[u] - f3[u] * f1[u];
          skn += k8[u];
        } else {
          s0 += r8[u] * f0[u];
          s1 += f0[u];
        }
        sr += r8[u];
        if (prefix ? (t + 1 == xnext) : (t == xnext)) {
          const int nch_ = prefix ? xnext - a : b - xnext;
          if (nch_ >= 2) {
            const float inv = 1.0f / (float)nch_;
            if (kside) {
              ck[ci * D + i] = s0 * inv;
            } else {
              const float beta = dm.beta_frac * sr * inv;
              cv[ci * D + i] = (s0 + beta * s1) / (sr + (float)nch_ * beta + dm.eps);
            }
          }
          if (lt == 0) {
            cn[ci] = (float)nch_;
            cR[ci] = sr;
            cKm[ci] = skn / (float)nch_;
          }
          ci += prefix ? 1 : -1;
          if (ci < 0 || ci >= nx) done = true;
          else xnext = xs[ci];
        }
      }
    }
  }
  __syncthreads();
  // ---- phase A2: coherence, multiplicity, representative position, RoPE(k) ----
  {
    const int wave = lt >> 6, lane = lt & 63;
    for (int c = wave; c < nx; c += GT / 64) {
      const int nch_ = (int)cn[c];
      if (nch_ < 2) continue;
      float ss = 0.f;
      for (int i = lane; i < D; i += 64) ss += ck[c * D + i] * ck[c * D + i];
      ss = wave_sum(ss);
      const int x0 = prefix ? a : xs[c];
      const int x1 = prefix ? xs[c] : b;
      const int p = round_half_even_mid((int)(a0 + x0), (int)(a0 + x1));
      const float coh = sqrtf(ss) / (cKm[c] + dm.eps);
      const float me = fminf(fmaxf((float)nch_ * coh * coh, 1.0f), (float)nch_);
      if (lane == 0) cMe[c] = me;
      for (int i = lane; i < H2; i += 64) {
        const float cc = cosT[(int64_t)p * H2 + i], sn = sinT[(int64_t)p * H2 + i];
        const float m1 = ck[c * D + i], m2 = ck[c * D + i + H2];
        ck[c * D + i] = m1 * cc - m2 * sn;
        ck[c * D + i + H2] = m2 * cc + m1 * sn;
      }
    }
  }
  __syncthreads();
  // ---- phase B: probe sweep (TPQ threads per probe, DPT dims each), loads 4 tokens ahead ----
  {
    const int q = lt / TPQ, sub = lt % TPQ;
    const int d0 = sub * DPT;
    if (q < dm.W && steps > 0) {
      float M[DPT];
#pragma unroll
      for (int k = 0; k < DPT; ++k) M[k] = 0.f;
      float Z = 0.f;
      int ci = prefix ? 0 : nx - 1;
      int xnext = xs[ci];
      bool done = false;
      for (int it0 = 0; it0 < steps && !done; it0 += 4) {
        float e4[4];
        float v4[4][DPT];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int t = t_first + step * min(it0 + u, steps - 1);
          e4[u] = U.sE[q * ES + t];
          lds_row<DPT>(U.sV + t * D + d0, v4[u]);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (done || it0 + u >= steps) break;
          const int t = t_first + step * (it0 + u);
          Z += e4[u];
#pragma unroll
          for (int k = 0; k < DPT; ++k) M[k] += e4[u] * v4[u][k];
          if (prefix ? (t + 1 == xnext) : (t == xnext)) {
            if ((int)cn[ci] >= 2) {
              float dot = 0.f;
#pragma unroll
              for (int k = 0; k < DPT; ++k) dot += qv[k] * ck[ci * D + d0 + k];
              dot += __shfl_xor(dot, 1, 64);
              dot += __shfl_xor(dot, 2, 64);
              const float zt = cMe[ci] * expf(dot * scale - m_q);
              float s1 = 0.f, s2 = 0.f;
#pragma unroll
              for (int k = 0; k < DPT; ++k) {
                const float df = M[k] - zt * cv[ci * D + d0 + k];
                s1 += df * df;
                s2 += M[k] * M[k];
              }
              s1 += __shfl_xor(s1, 1, 64);
              s1 += __shfl_xor(s1, 2, 64);
              s2 += __shfl_xor(s2, 1, 64);
              s2 += __shfl_xor(s2, 2, 64);
              const float dz = Z - zt;
              const float Dq = dm.lam_Z * dz * dz / (Z * Z + dm.eps) + dm.lam_M * s1 / (s2 + dm.eps);
              if (sub == 0) con[ci * WMAX + q] = (Z / zc_q) * Dq;
            }
            ci += prefix ? 1 : -1;
            if (ci < 0 || ci >= nx) done = true;
            else xnext = xs[ci];
          }
        }
      }
    }
  }
  __syncthreads();
  // ---- phase C: D = mean over probes (fixed order) ----
  if (lt < nx) {
    const int c = lt;
    float acc = 0.f;
    if ((int)cn[c] >= 2) {
      for (int qq = 0; qq < dm.W; ++qq) acc += con[c * WMAX + qq];
      acc /= (float)dm.W;
    }
    cD[c] = acc;
  }
  __syncthreads();
}

template <typename T, int D>
__global__ __launch_bounds__(BT) void k_build(Dims dm, int mode, const T* __restrict__ K, const T* __restrict__ V,
                                               const T* __restrict__ Q, const float* __restrict__ cosT,
                                               const float* __restrict__ sinT, const int32_t* __restrict__ slot_starts,
                                               const int32_t* __restrict__ n_slots, const float* __restrict__ kappa,
                                               TreeView tv) {
  using Lay = BuildLds<T, D>;
  constexpr bool BF = sizeof(T) == 2;
  constexpr int DPT = D / TPQ;
  constexpr int NW = BT / 64;
  extern __shared__ __align__(16) char smem[];
  Unit<T, D> U(smem);
  const int J = *n_slots;
  const int unit = blockIdx.x;
  const int lg = unit / dm.J_cap, j = unit % dm.J_cap;
  if (j >= J) return;
  const int l = lg / dm.G, g = lg % dm.G;
  const int64_t a0 = slot_starts[j];
  const int n = slot_starts[j + 1] - (int)a0;
  if (n < 1 || n > NMAX || a0 < 0 || a0 + n > dm.N_c) {   // malformed partition: refuse the unit
    if (threadIdx.x == 0) { atomicOr(tv.status, 2); tv.unit_nn[unit] = 0; }
    return;
  }
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const float scale = 1.0f / sqrtf((float)D);
  const int64_t base = (int64_t)lg * 2 * dm.N_c + 2 * a0;
  const uint32_t ord = (uint32_t)lg * (uint32_t)J + (uint32_t)j;
  const uint64_t theta = mode == BUILD_FULL ? 0ull : *tv.theta;
  int* cnt = U.xi + 192;       // node count
  {
    // resume from the node table: refine only nodes whose creating op reaches theta
    const int nn0 = tv.unit_nn[unit];
    const uint64_t Eadd = tv.add_E[unit];
    bool any = false;
    for (int i = tid; i < nn0; i += BT) {
      const int64_t sl = base + i;
      U.na[i] = tv.node_a[sl] - (int)a0; U.nn[i] = tv.node_n[sl]; U.nc[i] = tv.node_child[sl];
      U.np[i] = tv.node_parent[sl]; U.nch[i] = tv.node_nch[sl]; U.nk[i] = tv.node_kind[sl];
      U.ncut[i] = tv.node_cut[sl]; U.nD[i] = tv.node_D[sl]; U.nR[i] = tv.node_R[sl]; U.nU[i] = tv.sp_U[sl];
      const uint64_t ec = U.np[i] < 0 ? Eadd : tv.sp_E[base + U.np[i]];
      U.nE[i] = ec;
      any |= U.nch[i] == 0 && U.nn[i] >= 2 && ec >= theta && (mode != BUILD_ROOT_SPLIT || i == 0);
    }
    if (tid == 0) cnt[0] = nn0;
    if (!__syncthreads_or(any)) return;
  }
  const T* Kp = K + ((int64_t)lg * dm.T + a0) * D;
  const T* Vp = V + ((int64_t)lg * dm.T + a0) * D;
  const T* Qp = Q + ((int64_t)l * dm.H + (int64_t)g * dm.hpg) * dm.W * D;

  // ---- stage K, V (16-byte chunks; rows up to the last 16-token tile, zero past n) ----
  {
    constexpr int CH = 16 / (int)sizeof(T);          // elements per chunk
    constexpr int CPR = D / CH;                       // chunks per row
    const int rows = ((n + 15) / 16) * 16;
    for (int e = tid; e < rows * CPR; e += BT) {
      const int t = e / CPR, c = (e % CPR) * CH;
      uint4 kk = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
      if (t < n) {
        kk = *(const uint4*)(Kp + (int64_t)t * D + c);
        vv = *(const uint4*)(Vp + (int64_t)t * D + c);
      }
      T* dk = U.sK + t * Lay::LDK + c;
      if constexpr (sizeof(T) == 2) {                 // LDK rows are 8-byte aligned for bf16
        uint2* d2 = (uint2*)dk;
        d2[0] = make_uint2(kk.x, kk.y);
        d2[1] = make_uint2(kk.z, kk.w);
      } else {
        const float* kf = (const float*)&kk;
        for (int h = 0; h < 4; ++h) dk[h] = kf[h];
      }
      *(uint4*)(U.sV + t * D + c) = vv;
    }
  }
  __syncthreads();

  // ---- probe exponentials e_{q,t} (matrix cores; probe q = window query q of
  // head q mod |H(g)|).  A = probe rows, B = keys; each lane supplies a quarter
  // row (D/4 consecutive dims) per operand. ----
  {
    constexpr int QE = D / 4;
    const int i16 = lane & 15, g4 = lane >> 4;
    const int n_pt = (dm.W + 15) / 16, n_tt = (n + 15) / 16;
    for (int pi = wave; pi < n_pt * n_tt; pi += NW) {
      const int pt = pi % n_pt, tt = pi / n_pt;
      const int up = 16 * pt + i16;
      const int uq = up < dm.W ? up : 0;
      const T* qr = Qp + ((int64_t)(uq % dm.hpg) * dm.W + uq) * D + QE * g4;
      const T* kr = U.sK + (16 * tt + i16) * Lay::LDK + QE * g4;
      float mqr[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int u2 = 16 * pt + 4 * g4 + r;
        mqr[r] = u2 < dm.W ? tv.probe_m[(int64_t)lg * dm.W + u2] : 0.f;
      }
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      if constexpr (BF) {
#pragma unroll
        for (int s2 = 0; s2 < QE / 4; ++s2) {
          const uint2 qa = *(const uint2*)(qr + 4 * s2);
          const uint2 kb = *(const uint2*)(kr + 4 * s2);
          s16x4 av, bv;
          av[0] = (short)(qa.x & 0xffffu); av[1] = (short)(qa.x >> 16); av[2] = (short)(qa.y & 0xffffu); av[3] = (short)(qa.y >> 16);
          bv[0] = (short)(kb.x & 0xffffu); bv[1] = (short)(kb.x >> 16); bv[2] = (short)(kb.y & 0xffffu); bv[3] = (short)(kb.y >> 16);
          acc = mfma_bf16_16x16x16(av, bv, acc);
        }
      } else {
#pragma unroll
        for (int s2 = 0; s2 < QE; ++s2) acc = mfma_f32_16x16x4(((const float*)qr)[s2], ((const float*)kr)[s2], acc);
      }
      const int t = 16 * tt + i16;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int u2 = 16 * pt + 4 * g4 + r;
        if (u2 < dm.W && t < n) U.sE[u2 * ES + t] = expf(acc[r] * scale - mqr[r]);
      }
    }
  }
  // ---- token values, probe masses, curvature, key norms ----
  if (tid < n) {
    const int t = tid;
    U.sR[t] = tv.tok_R[(int64_t)lg * dm.N_c + a0 + t];
    U.sA[t] = tv.tok_A[(int64_t)lg * dm.N_c + a0 + t];
    U.sKap[t] = kappa[a0 + t];
    float kn = 0.f;
    for (int c = 0; c < D; ++c) {
      const float x = ldf(U.sK, t * Lay::LDK + c);
      kn += x * x;
    }
    U.sKn[t] = sqrtf(kn);
  }
  __syncthreads();

  // ---- probe registers for the sweeps (same probe in both groups) ----
  const int lt = tid % GT;
  const int q = lt / TPQ;
  float qv[DPT];
  float m_q = 0.f, zc_q = 1.f;
  if (q < dm.W) {
    const int hl = q % dm.hpg;
    const T* qr = Qp + ((int64_t)hl * dm.W + q) * D + (lt % TPQ) * DPT;
#pragma unroll
    for (int k = 0; k < DPT; ++k) qv[k] = ldf(qr, k);
    m_q = tv.probe_m[(int64_t)lg * dm.W + q];
    zc_q = tv.probe_ZC[(int64_t)lg * dm.W + q];
  } else {
#pragma unroll
    for (int k = 0; k < DPT; ++k) qv[k] = 0.f;
  }

  // ---- root ----
  int* XL = U.xi;              // [0..31]
  int* XR = U.xi + 32;         // [32..63]
  int* XB = U.xi + 64;         // [64..95] binary cuts
  int* meta = U.xi + 96;       // nXL, nXR, nXB, p, kmin bits, kmax bits, index of p in XL, of p+1 in XR
  float* cRL = U.gcs(0, 1);
  float* cDL = U.gcs(0, 5);
  float* cRR = U.gcs(1, 1);
  float* cDR = U.gcs(1, 5);
  const float w = tv.omega[lg];

  // ---- top-down refinement in BFS order ----
  for (int head = 0;; ++head) {
    __syncthreads();
    const int count = cnt[0];
    if (head >= count || (mode == BUILD_ROOT_SPLIT && head > 0)) break;
    const int a = U.na[head], nv = U.nn[head], b = a + nv;
    if (nv < 2 || U.nch[head] > 0) continue;                  // leaf, or refined by an earlier pass
    if (mode != BUILD_FULL && U.nE[head] < theta) continue;    // cannot reach the auction's cut
    const float Dv = U.nD[head];
    if (nv == 2) {
      if (tid == 0) {
        const int c0 = count;
        U.nc[head] = c0; U.nch[head] = 2; U.nk[head] = 1; U.ncut[head] = (int)a0 + a + 1;
        for (int k = 0; k < 2; ++k) {
          U.na[c0 + k] = a + k; U.nn[c0 + k] = 1; U.nc[c0 + k] = -1; U.np[c0 + k] = head;
          U.nch[c0 + k] = 0; U.nk[c0 + k] = 0; U.ncut[c0 + k] = -1;
          U.nD[c0 + k] = 0.f; U.nR[c0 + k] = U.sR[a + k];
        }
        cnt[0] = count + 2;
        if (mode != BUILD_FULL) {
          const float Us = utility(split_gain(w, U.nR[head], Dv, U.nD[c0] + U.nD[c0 + 1]), 1);
          const uint64_t k = op_key(Us, ord * 256u + 1u + (uint32_t)head);
          const uint64_t E = k < U.nE[head] ? k : U.nE[head];
          U.nU[head] = Us;
          U.nE[c0] = E; U.nE[c0 + 1] = E;
        }
      }
      continue;
    }
    // candidate flags over cut positions xi in (a, b)
    for (int t = tid; t < NMAX; t += BT) U.flag[t] = 0;
    __syncthreads();
    if (tid < nv - 1) {
      const int t = a + tid;                     // curvature position t -> cut t + 1
      const float kt = U.sKap[t];
      int rank = 0;
      for (int t2 = a; t2 <= b - 2; ++t2) {
        const float k2 = U.sKap[t2];
        rank += (k2 > kt) || (k2 == kt && t2 < t);
      }
      if (rank < dm.k_curv) U.flag[t + 1 - a] = 1;
    }
    if (tid == BT - 1) U.flag[nv / 2] = 1;      // midpoint a + floor(n/2)
    // curvature range and extraction token (wave 0)
    if (wave == 0) {
      float kmn = INFINITY, kmx = -INFINITY, best = -INFINITY;
      int bi = 0x7fffffff;
      for (int t = a + lane; t < b; t += 64) {
        const float k = U.sKap[t];
        kmn = fminf(kmn, k);
        kmx = fmaxf(kmx, k);
        const float am = U.sA[t];
        if (am > best || (am == best && t < bi)) { best = am; bi = t; }
      }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        kmn = fminf(kmn, __shfl_xor(kmn, o, 64));
        kmx = fmaxf(kmx, __shfl_xor(kmx, o, 64));
        const float b2 = __shfl_xor(best, o, 64);
        const int i2 = __shfl_xor(bi, o, 64);
        if (b2 > best || (b2 == best && i2 < bi)) { best = b2; bi = i2; }
      }
      if (lane == 0) {
        meta[3] = bi;
        meta[4] = __float_as_int(kmn);
        meta[5] = __float_as_int(kmx);
      }
    }
    __syncthreads();
    // binary cuts XB (ascending) by ballot over the flags, then the prefix list
    // XL = XB + {p} (if p > a) and suffix list XR = XB + {p+1} (if p+1 < b)
    int* posL = U.xi + 128;      // index of XB[k] in XL
    int* posR = U.xi + 160;      // index of XB[k] in XR
    if (wave == 0) {
      const bool f0 = lane >= 1 && lane < nv && U.flag[lane];
      const bool f1 = 64 + lane < nv && U.flag[64 + lane];
      const uint64_t m0 = __ballot(f0), m1 = __ballot(f1);
      const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
      const int n0 = __popcll(m0);
      if (f0) XB[__popcll(m0 & below)] = a + lane;
      if (f1) XB[n0 + __popcll(m1 & below)] = a + 64 + lane;
      if (lane == 0) meta[2] = n0 + __popcll(m1);
    }
    __syncthreads();
    if (wave == 0) {
      const int nb = meta[2], p = meta[3];
      const bool on = lane < nb;
      const int xk = on ? XB[lane] : 0x7fffffff;
      const bool useP = p > a, useQ = p + 1 < b;
      const uint64_t lessP = __ballot(on && xk < p), eqP = __ballot(on && xk == p);
      const uint64_t lessQ = __ballot(on && xk < p + 1), eqQ = __ballot(on && xk == p + 1);
      const bool insL = useP && eqP == 0ull, insR = useQ && eqQ == 0ull;
      if (on) {
        const int pl = lane + ((insL && xk > p) ? 1 : 0);
        const int pr = lane + ((insR && xk > p + 1) ? 1 : 0);
        XL[pl] = xk; posL[lane] = pl;
        XR[pr] = xk; posR[lane] = pr;
      }
      if (lane == 0) {
        const int cp = __popcll(lessP), cq = __popcll(lessQ);
        if (insL) XL[cp] = p;
        if (insR) XR[cq] = p + 1;
        meta[0] = nb + (insL ? 1 : 0);
        meta[1] = nb + (insR ? 1 : 0);
        meta[6] = useP ? cp : -1;         // index of p in XL ([a, p))
        meta[7] = useQ ? cq : -1;         // index of p + 1 in XR ([p+1, b))
      }
    }
    __syncthreads();
    const int nl = meta[0], nr = meta[1], nb = meta[2], p = meta[3];
    sweep2<T, D>(U, dm, a, b, XL, nl, XR, nr, a0, cosT, sinT, qv, m_q, zc_q, scale);
    // scores (fp32): best binary cut by a wave-0 argmax (smaller cut wins ties),
    // then the extraction score and the append by lane 0
    if (wave == 0) {
      const float kmn = __int_as_float(meta[4]), kmx = __int_as_float(meta[5]);
      const float kr = kmx - kmn;
      float best = -INFINITY;
      int bk = 0x7fffffff;
      if (lane < nb) {
        const int x = XB[lane];
        const float kh = kr > 0.f ? (U.sKap[x - 1] - kmn) / kr : 0.f;
        best = ((Dv - cDL[posL[lane]]) - cDR[posR[lane]]) + dm.lam_kappa * kh;
        bk = lane;
      }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        const float b2 = __shfl_xor(best, o, 64);
        const int k2 = __shfl_xor(bk, o, 64);
        if (b2 > best || (b2 == best && k2 < bk)) { best = b2; bk = k2; }
      }
      if (lane == 0) {
        const int iL = meta[6], iR = meta[7];
        float dsum = 0.f;
        int nkid = 1;
        if (p > a) { dsum += cDL[iL]; ++nkid; }
        if (p + 1 < b) { dsum += cDR[iR]; ++nkid; }
        const float gext = (Dv - dsum) / (float)(nkid - 1);
        const int c0 = count;
        U.nc[head] = c0;
        int c = c0;
        if (best >= gext) {
          const int bx = XB[bk];
          U.nch[head] = 2; U.nk[head] = 1; U.ncut[head] = (int)a0 + bx;
          U.na[c] = a; U.nn[c] = bx - a; U.nD[c] = cDL[posL[bk]]; U.nR[c] = cRL[posL[bk]]; ++c;
          U.na[c] = bx; U.nn[c] = b - bx; U.nD[c] = cDR[posR[bk]]; U.nR[c] = cRR[posR[bk]]; ++c;
        } else {
          U.nch[head] = nkid; U.nk[head] = 2; U.ncut[head] = (int)a0 + p;
          if (p > a) { U.na[c] = a; U.nn[c] = p - a; U.nD[c] = cDL[iL]; U.nR[c] = cRL[iL]; ++c; }
          U.na[c] = p; U.nn[c] = 1; U.nD[c] = 0.f; U.nR[c] = U.sR[p]; ++c;
          if (p + 1 < b) { U.na[c] = p + 1; U.nn[c] = b - p - 1; U.nD[c] = cDR[iR]; U.nR[c] = cRR[iR]; ++c; }
        }
        for (int k = c0; k < c; ++k) { U.nc[k] = -1; U.np[k] = head; U.nch[k] = 0; U.nk[k] = 0; U.ncut[k] = -1; }
        cnt[0] = c;
        if (mode != BUILD_FULL) {
          float sd = 0.f;
          for (int k = c0; k < c; ++k) sd += U.nD[k];
          const float Us = utility(split_gain(w, U.nR[head], Dv, sd), c - c0 - 1);
          const uint64_t kk = op_key(Us, ord * 256u + 1u + (uint32_t)head);
          const uint64_t E = kk < U.nE[head] ? kk : U.nE[head];
          U.nU[head] = Us;
          for (int k = c0; k < c; ++k) U.nE[k] = E;
        }
      }
    }
  }
  __syncthreads();
  // ---- write the node table ----
  const int count = cnt[0];
  for (int i = tid; i < 2 * n; i += BT) {
    const int64_t sl = base + i;
    if (i < count) {
      tv.node_a[sl] = (int32_t)a0 + U.na[i];
      tv.node_n[sl] = U.nn[i];
      tv.node_child[sl] = U.nc[i];
      tv.node_parent[sl] = U.np[i];
      tv.node_nch[sl] = (uint8_t)U.nch[i];
      tv.node_kind[sl] = (uint8_t)U.nk[i];
      tv.node_cut[sl] = U.ncut[i];
      tv.node_D[sl] = U.nD[i];
      tv.node_R[sl] = U.nR[i];
      if (mode != BUILD_FULL) {          // keys of the Splits known so far (refined nodes)
        const int c = U.nch[i];
        if (c > 0) {
          const uint64_t k = op_key(U.nU[i], ord * 256u + 1u + (uint32_t)i);
          tv.sp_U[sl] = U.nU[i];
          tv.sp_E[sl] = k < U.nE[i] ? k : U.nE[i];
          tv.sp_cost[sl] = (uint8_t)(c - 1);
        } else {
          tv.sp_U[sl] = 0.f;
          tv.sp_E[sl] = 0;
          tv.sp_cost[sl] = 0;
        }
        tv.sp_exec[sl] = 0;
      }
    } else {
      tv.sp_cost[sl] = 0;
      tv.sp_E[sl] = 0;
      tv.sp_exec[sl] = 0;
    }
  }
  if (tid == 0) tv.unit_nn[unit] = count;
}

hipError_t launch_build(const Dims& dm, int lds_bytes, int mode, const void* K, const void* V, const void* Q,
                        const float* cosT, const float* sinT, const int32_t* slot_starts, const int32_t* n_slots,
                        const float* kappa, const TreeView& tv, hipStream_t st) {
  const dim3 grid((unsigned)((int64_t)dm.L * dm.G * dm.J_cap));
#define GKV_LAUNCH_BUILD(TT, DD)                                                                           \
  do {                                                                                                     \
    auto fn = k_build<TT, DD>;                                                                             \
    hipError_t e0 = hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes); \
    if (e0 != hipSuccess) return e0;                                                                       \
    hipLaunchKernelGGL(fn, grid, dim3(BT), lds_bytes, st, dm, mode, (const TT*)K, (const TT*)V, (const TT*)Q, cosT, \
                       sinT, slot_starts, n_slots, kappa, tv);                                             \
  } while (0)
  if (dm.dtype == GRACEKV_BF16) {
    if (dm.d == 128) GKV_LAUNCH_BUILD(uint16_t, 128); else GKV_LAUNCH_BUILD(uint16_t, 64);
  } else {
    if (dm.d == 128) GKV_LAUNCH_BUILD(float, 128); else GKV_LAUNCH_BUILD(float, 64);
  }
#undef GKV_LAUNCH_BUILD
  return hipGetLastError();
}

}  // namespace gkv
