// Decode-time attention over the packed cache (App. A.3 eq:app_decode_logit;
// App. A.5 "Frontier updates and physical packing").
//
// For every layer l and query head h (KV head g = h / hpg) one decode query
// attends to the packed entries of (l, g), with logits q.k~ / sqrt(d) +
// log m_eff, and to the window rows N_ctx .. T-1 of K, V (kept exactly,
// log m_eff = 0), and returns the softmax-weighted mean of the values.
//
// The work is a stream over the packed rows, bound by HBM: every entry's key
// and value are read once for all query heads of its group.
//   * grid (P, L*G), 256 threads: workgroup p of (l, g) takes the p-th of P
//     contiguous ranges of the row.  One entry sits on D/8 lanes (eight dims
//     each), so a wave reads whole rows, the next entry's rows in flight while
//     the current one is folded in; each such lane group keeps a base-2
//     online-softmax state per query head (running max, sum, its eight output
//     dims).  The lane groups of a wave merge through row-swap permutations,
//     the four waves through LDS; the partial state goes to the workspace.
//   * k_decode_combine, one workgroup per (l, g), one thread per (query head,
//     dim): merges the P partial states and writes the normalised output.  (A
//     last-arriving workgroup could merge them in the same launch, but the
//     device-scope fences that needs write back and invalidate the L2 of the
//     XCD on this chip, which costs far more than a second launch.)
#include <mutex>

#include "common.h"

namespace gkv {

constexpr int DEC_T = 256;
constexpr int DEC_W = DEC_T / 64;
constexpr int DEC_PMAX = 64;

// workspace: partial states [L*G][P][hpg] (max, sum) as float2, then
// [L*G][P][hpg][d] fp32
static size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }
size_t decode_ws_bytes(const Dims& dm, int P) {
  const size_t n = (size_t)dm.L * dm.G * P * dm.hpg;
  return al256(n * 8) + n * dm.d * 4;
}

int decode_parts(const Dims& dm) {
  const int64_t per = dm.B_total / ((int64_t)dm.L * dm.G) + (dm.T - dm.N_ctx);
  int64_t P = (per + 127) / 128;
  return (int)(P < 1 ? 1 : (P > DEC_PMAX ? DEC_PMAX : P));
}

// raw eight values of a row (held while the previous entry is folded in)
template <typename T> struct Raw8;
template <> struct Raw8<uint16_t> {
  uint4 u;
  __device__ __forceinline__ void load(const uint16_t* p) { u = *(const uint4*)p; }
  __device__ __forceinline__ void get(float* x) const {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(w[i] << 16);
      x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
};
template <> struct Raw8<float> {
  float4 a, b;
  __device__ __forceinline__ void load(const float* p) { a = *(const float4*)p; b = *(const float4*)(p + 4); }
  __device__ __forceinline__ void get(float* x) const {
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
  }
};

// eight consecutive values of a row as fp32
__device__ __forceinline__ void load8(const uint16_t* p, float* x) {
  const uint4 u = *(const uint4*)p;
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void load8(const float* p, float* x) {
  const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}

// sum over the D/8 lanes of one entry (16-lane rows for d = 128, 8-lane halves for d = 64)
template <int D>
__device__ __forceinline__ float entry_sum(float v) {
  if constexpr (D == 128) {
    return row_sum16(v);
  } else {
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xf, 0xf, false));   // lane ^ 1
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xf, 0xf, false));   // lane ^ 2
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xf, 0xf, false));  // half-row mirror
    return v;
  }
}

// maximum over the lane groups of a wave that hold the same dims (lanes l,
// l + D/8, ...), returned to all of them
template <int D>
__device__ __forceinline__ float group_max(float v) {
  if constexpr (D == 64) {   // the two 8-lane halves of a row: rotate the row by 8
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xf, 0xf, false)));
  }
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1]));
}
template <int D>
__device__ __forceinline__ float group_sum(float v) {
  if constexpr (D == 64) v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xf, 0xf, false));
  return col_sum4(v);
}

template <typename T, int D, int HPG>
__global__ __launch_bounds__(DEC_T) void k_decode(Dims dm, int P, const T* __restrict__ q,
                                                  const int64_t* __restrict__ offsets, const T* __restrict__ Kout,
                                                  const T* __restrict__ Vout, const float* __restrict__ logm,
                                                  const T* __restrict__ K, const T* __restrict__ V,
                                                  float2* __restrict__ pml, float* __restrict__ po) {
  constexpr int LPE = D / 8;                  // lanes per entry
  constexpr int EPW = 64 / LPE;               // entries per wave step
  constexpr float LOG2E = 1.44269504088896341f;
  __shared__ float sM[DEC_W][HPG], sS[DEC_W][HPG];
  __shared__ float sO[DEC_W][HPG][D];
  const int lg = blockIdx.y, p = blockIdx.x;
  const int l = lg / dm.G, g = lg % dm.G;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int sub = lane % LPE, row = lane / LPE;
  // the (l, g) row: packed entries [o0, o1) (clamped into the cache), then the window rows
  int64_t o0 = offsets[lg], o1 = offsets[lg + 1];
  o0 = o0 < 0 ? 0 : (o0 > dm.B_total ? dm.B_total : o0);
  o1 = o1 < o0 ? o0 : (o1 > dm.B_total ? dm.B_total : o1);
  const int64_t cnt = o1 - o0, n = cnt + (dm.T - dm.N_ctx);
  const int64_t e0 = n * p / P, e1 = n * (p + 1) / P;
  // queries of the group, dims 8 sub .. + 7, with the logit scale in base-2 units
  const float sc2 = LOG2E / sqrtf((float)D);
  float qv[HPG][8];
#pragma unroll
  for (int h = 0; h < HPG; ++h) {
    load8(q + ((int64_t)l * dm.H + (int64_t)g * HPG + h) * D + 8 * sub, qv[h]);
#pragma unroll
    for (int j = 0; j < 8; ++j) qv[h][j] *= sc2;
  }
  float m[HPG], s[HPG], o[HPG][8];
#pragma unroll
  for (int h = 0; h < HPG; ++h) {
    m[h] = -INFINITY;
    s[h] = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) o[h][j] = 0.f;
  }
  // entry e of the row: packed row o0 + e, or window row N_ctx + e - cnt
  auto locate = [&](int64_t e, const T*& kr, const T*& vr, float& lm) {
    if (e < cnt) {
      kr = Kout + (o0 + e) * D;
      vr = Vout + (o0 + e) * D;
      lm = logm[o0 + e] * LOG2E;
    } else {
      const int64_t t = dm.N_ctx + (e - cnt);
      kr = K + ((int64_t)lg * dm.T + t) * D;
      vr = V + ((int64_t)lg * dm.T + t) * D;
      lm = 0.f;
    }
  };
  // wave-uniform trip count; a lane group past e1 contributes nothing
  constexpr int64_t STEP = (int64_t)DEC_W * EPW;
  Raw8<T> kn, vn;
  float lmn = 0.f;
  {
    const int64_t e = e0 + (int64_t)w * EPW + row;
    const T* kr;
    const T* vr;
    locate(e < e1 ? e : e0, kr, vr, lmn);
    if (e0 < e1) { kn.load(kr + 8 * sub); vn.load(vr + 8 * sub); }
  }
  for (int64_t eb = e0 + (int64_t)w * EPW; eb < e1; eb += STEP) {
    const bool on = eb + row < e1;
    float kx[8], vx[8];
    kn.get(kx);
    vn.get(vx);
    const float lm = lmn;
    if (eb + STEP < e1) {                     // the next entry of this lane group, in flight
      const int64_t e = eb + STEP + row;
      const T* kr;
      const T* vr;
      locate(e < e1 ? e : e0, kr, vr, lmn);
      kn.load(kr + 8 * sub);
      vn.load(vr + 8 * sub);
    }
#pragma unroll
    for (int h = 0; h < HPG; ++h) {
      float x = 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) x += qv[h][j] * kx[j];
      x = entry_sum<D>(x) + lm;
      if (on) {
        const float mn = fmaxf(m[h], x);
        const float c = __builtin_amdgcn_exp2f(m[h] - mn);
        const float pe = __builtin_amdgcn_exp2f(x - mn);
        s[h] = s[h] * c + pe;
#pragma unroll
        for (int j = 0; j < 8; ++j) o[h][j] = o[h][j] * c + pe * vx[j];
        m[h] = mn;
      }
    }
  }
  // merge the lane groups of the wave, then the waves
#pragma unroll
  for (int h = 0; h < HPG; ++h) {
    const float M = group_max<D>(m[h]);
    const float c = m[h] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m[h] - M);
    const float S = group_sum<D>(s[h] * c);
    float oo[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) oo[j] = group_sum<D>(o[h][j] * c);
    if (row == 0) {
      if (sub == 0) { sM[w][h] = M; sS[w][h] = S; }
#pragma unroll
      for (int j = 0; j < 8; ++j) sO[w][h][8 * sub + j] = oo[j];
    }
  }
  __syncthreads();
  const int64_t part = ((int64_t)lg * P + p) * HPG;
  for (int i = tid; i < HPG * D; i += DEC_T) {
    const int h = i / D, dd = i % D;
    float M = -INFINITY;
#pragma unroll
    for (int w2 = 0; w2 < DEC_W; ++w2) M = fmaxf(M, sM[w2][h]);
    float S = 0.f, O = 0.f;
#pragma unroll
    for (int w2 = 0; w2 < DEC_W; ++w2) {
      const float c = sM[w2][h] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sM[w2][h] - M);
      S += sS[w2][h] * c;
      O += sO[w2][h][dd] * c;
    }
    po[(part + h) * D + dd] = O;
    if (dd == 0) pml[part + h] = make_float2(M, S);
  }
}

template <int D>
__global__ __launch_bounds__(512) void k_decode_combine(Dims dm, int P, const float2* __restrict__ pml,
                                                        const float* __restrict__ po, float* __restrict__ out) {
  const int lg = blockIdx.x;
  const int l = lg / dm.G, g = lg % dm.G;
  for (int i = threadIdx.x; i < dm.hpg * D; i += blockDim.x) {
    const int h = i / D, dd = i % D;
    const int64_t row0 = (int64_t)lg * P * dm.hpg + h;
    float M = -INFINITY;
#pragma unroll 4
    for (int q2 = 0; q2 < P; ++q2) M = fmaxf(M, pml[row0 + (int64_t)q2 * dm.hpg].x);
    float S = 0.f, O = 0.f;
#pragma unroll 4
    for (int q2 = 0; q2 < P; ++q2) {
      const int64_t k = row0 + (int64_t)q2 * dm.hpg;
      const float2 ms = pml[k];
      const float c = ms.x == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ms.x - M);
      S += ms.y * c;
      O += po[k * D + dd] * c;
    }
    out[((int64_t)l * dm.H + (int64_t)g * dm.hpg + h) * D + dd] = S > 0.f ? O / S : 0.f;
  }
}

// Fixed device scratch of the allocation-free entry point: the partial softmax
// states of the split over entries.  Every GPU the library runs on holds its own
// copy at its own address until the process ends; host code never uses the
// array's name as an address, only the pointer hipGetSymbolAddress returns
// for the current device (scratch_on_device).
static __device__ __align__(256) char scratch[GRACEKV_DECODE_SCRATCH_BYTES];

static hipError_t scratch_on_device(void** out) {
  constexpr int NDEV = 64;
  static void* ptr[NDEV] = {nullptr};
  static std::mutex mu;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= NDEV) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    ptr[dev] = p;
  }
  *out = ptr[dev];
  return hipSuccess;
}

hipError_t launch_decode_noalloc(const Dims& dm, const void* q, const int64_t* offsets, const void* K_out,
                                 const void* V_out, const float* logm_out, const void* K, const void* V, float* out,
                                 hipStream_t st) {
  if (decode_ws_bytes(dm, decode_parts(dm)) > (size_t)GRACEKV_DECODE_SCRATCH_BYTES) return hipErrorInvalidValue;
  void* ws = nullptr;
  const hipError_t e = scratch_on_device(&ws);
  if (e != hipSuccess) return e;
  return launch_decode(dm, q, offsets, K_out, V_out, logm_out, K, V, out, ws, st);
}

hipError_t launch_decode(const Dims& dm, const void* q, const int64_t* offsets, const void* K_out, const void* V_out,
                         const float* logm_out, const void* K, const void* V, float* out, void* ws,
                         hipStream_t st) {
  const int P = decode_parts(dm);
  const size_t n = (size_t)dm.L * dm.G * P * dm.hpg;
  float2* pml = (float2*)ws;
  float* po = (float*)((char*)ws + al256(n * 8));
  const dim3 grid((unsigned)P, (unsigned)(dm.L * dm.G));
#define GKV_DEC(TT, DD, HH)                                                                                    \
  hipLaunchKernelGGL((k_decode<TT, DD, HH>), grid, dim3(DEC_T), 0, st, dm, P, (const TT*)q, offsets,          \
                     (const TT*)K_out, (const TT*)V_out, logm_out, (const TT*)K, (const TT*)V, pml, po)
#define GKV_DEC_H(TT, DD)                                                                                      \
  do {                                                                                                         \
    if (dm.hpg == 1) GKV_DEC(TT, DD, 1); else if (dm.hpg == 2) GKV_DEC(TT, DD, 2);                             \
    else if (dm.hpg == 4) GKV_DEC(TT, DD, 4); else if (dm.hpg == 8) GKV_DEC(TT, DD, 8);                       \
    else return hipErrorInvalidValue;                                                                          \
  } while (0)
  if (dm.dtype == GRACEKV_BF16) {
    if (dm.d == 128) GKV_DEC_H(uint16_t, 128); else if (dm.d == 64) GKV_DEC_H(uint16_t, 64);
    else return hipErrorInvalidValue;
  } else {
    if (dm.d == 64) GKV_DEC_H(float, 64); else return hipErrorInvalidValue;
  }
#undef GKV_DEC_H
#undef GKV_DEC
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 cb((unsigned)(dm.hpg * dm.d < 512 ? dm.hpg * dm.d : 512));
  if (dm.d == 128)
    hipLaunchKernelGGL(k_decode_combine<128>, dim3(dm.L * dm.G), cb, 0, st, dm, P, pml, po, out);
  else
    hipLaunchKernelGGL(k_decode_combine<64>, dim3(dm.L * dm.G), cb, 0, st, dm, P, pml, po, out);
  return hipGetLastError();
}

}  // namespace gkv
