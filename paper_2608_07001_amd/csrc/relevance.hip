// Relevance row statistics (pass 1 of the direct-relevance softmax).
//
// App. A.4 eq:app_attention_probability normalises each window query's
// attention over its complete causal range V(u) = [0, N_ctx + u]; the tree
// build (pass 2) needs, per row r = (query head, window position), the
// running maximum m_V and the partition Z_V over V(u), and over the
// compressible context C = [0, N_c) the maximum m_C and partition Z_C.  The
// probe shift of the distortion (read as the maximum logit over C) and
// Z_q(C) are the (m_C, Z_C) of the probe's row.  The per-(l, g) normaliser of
// eq:app_direct_relevance follows exactly:
//   sum_{t in C} s_t = sum_r exp(m_C - m_V) Z_C / Z_V.
//
// K5a: grid (chunks of T, L*G, row groups of 256).  Each workgroup stages
// 64-token sub-chunks of K in LDS and forms 16x16 logit tiles with MFMA
// (bf16 inputs: exact products, fp32 accumulation); each lane keeps online
// (max, sum-exp) pairs for its 4 rows, merged across lanes at the end.
// K5b: per (l, g), merge the chunk partials in order and reduce S.
#include "common.h"

namespace gkv {

constexpr int RS_SUB = 64;      // tokens per LDS sub-chunk
constexpr int RS_CHUNK = 2048;  // tokens per workgroup

int rowstats_chunks(const Dims& dm) { return (int)((dm.T + RS_CHUNK - 1) / RS_CHUNK); }

template <typename T> struct KPad;
template <> struct KPad<uint16_t> { static constexpr int v = 4; };
template <> struct KPad<float> { static constexpr int v = 1; };

template <typename T, int D>
__device__ __forceinline__ f32x4 logit_tile(const T* qrow_unused, const T* sK, int ldk, int tok0, int lane,
                                            const void* qf, f32x4 acc);

template <typename T, int D>
__global__ __launch_bounds__(256) void k_rowstats(Dims dm, const T* __restrict__ K, const T* __restrict__ Q,
                                                  float4* __restrict__ partial, int nchunk) {
  constexpr bool BF = sizeof(T) == 2;
  constexpr int KS = BF ? D / 16 : D / 4;         // MFMA k-steps
  constexpr int LDK = D + KPad<T>::v;
  __shared__ T sK[RS_SUB * LDK];

  const int ck = blockIdx.x, lg = blockIdx.y, rg = blockIdx.z;
  const int l = lg / dm.G, g = lg % dm.G;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t t_begin = (int64_t)ck * RS_CHUNK;
  const int64_t t_end = min(dm.T, t_begin + RS_CHUNK);
  const T* Kp = K + (int64_t)lg * dm.T * D;
  const T* Qp = Q + ((int64_t)l * dm.H + (int64_t)g * dm.hpg) * dm.W * D;
  const float scale = 1.0f / sqrtf((float)D);

  // this wave's 4 row tiles
  int rt0 = rg * 16 + wave * 4;
  bool tile_ok[4];
  // Q fragments in registers
  s16x4 qb[4][BF ? KS : 1];
  float qf[4][BF ? 1 : KS];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    int rt = rt0 + k;
    tile_ok[k] = rt * 16 < dm.rows;
    int row = rt * 16 + (lane & 15);
    bool rok = row < dm.rows;
    const T* qr = Qp + (int64_t)(rok ? row : 0) * D;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      if constexpr (BF) {
        s16x4 v;
        const uint16_t* q16 = (const uint16_t*)qr + s * 16 + 4 * (lane >> 4);
        v[0] = rok ? (short)q16[0] : 0;
        v[1] = rok ? (short)q16[1] : 0;
        v[2] = rok ? (short)q16[2] : 0;
        v[3] = rok ? (short)q16[3] : 0;
        qb[k][s] = v;
      } else {
        qf[k][s] = rok ? ((const float*)qr)[s * 4 + (lane >> 4)] : 0.f;
      }
    }
  }
  float mV[4][4], zV[4][4], mC[4][4], zC[4][4];
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int i = 0; i < 4; ++i) { mV[k][i] = -INFINITY; zV[k][i] = 0.f; mC[k][i] = -INFINITY; zC[k][i] = 0.f; }

  for (int64_t s0 = t_begin; s0 < t_end; s0 += RS_SUB) {
    __syncthreads();
    // stage K[s0 .. s0+SUB) (zero beyond the chunk)
    for (int e = threadIdx.x; e < RS_SUB * D; e += 256) {
      int tr = e / D, c = e % D;
      int64_t t = s0 + tr;
      sK[tr * LDK + c] = (t < t_end) ? Kp[t * D + c] : (T)0;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (!tile_ok[k]) continue;
#pragma unroll
      for (int tt = 0; tt < RS_SUB / 16; ++tt) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        const T* kr = sK + (tt * 16 + (lane & 15)) * LDK;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          if constexpr (BF) {
            const uint16_t* k16 = (const uint16_t*)kr + s * 16 + 4 * (lane >> 4);
            s16x4 b;
            b[0] = (short)k16[0]; b[1] = (short)k16[1]; b[2] = (short)k16[2]; b[3] = (short)k16[3];
            acc = mfma_bf16_16x16x16(qb[k][s], b, acc);
          } else {
            acc = mfma_f32_16x16x4(qf[k][s], ((const float*)kr)[s * 4 + (lane >> 4)], acc);
          }
        }
        const int64_t t = s0 + tt * 16 + (lane & 15);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = (rt0 + k) * 16 + 4 * (lane >> 4) + i;
          const int u = row % dm.W;
          const float x = acc[i] * scale;
          const bool vis = (t < t_end) && (t <= dm.N_ctx + u) && (row < dm.rows);
          const bool inC = vis && (t < dm.N_c);
          if (vis) {
            if (x > mV[k][i]) { zV[k][i] = zV[k][i] * expf(mV[k][i] - x) + 1.f; mV[k][i] = x; }
            else zV[k][i] += expf(x - mV[k][i]);
          }
          if (inC) {
            if (x > mC[k][i]) { zC[k][i] = zC[k][i] * expf(mC[k][i] - x) + 1.f; mC[k][i] = x; }
            else zC[k][i] += expf(x - mC[k][i]);
          }
        }
      }
    }
  }
  // merge across the 16 lanes holding the same rows
#pragma unroll
  for (int k = 0; k < 4; ++k) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        float m2 = __shfl_xor(mV[k][i], o, 64), z2 = __shfl_xor(zV[k][i], o, 64);
        lse_merge(mV[k][i], zV[k][i], m2, z2);
        m2 = __shfl_xor(mC[k][i], o, 64);
        z2 = __shfl_xor(zC[k][i], o, 64);
        lse_merge(mC[k][i], zC[k][i], m2, z2);
      }
      const int row = (rt0 + k) * 16 + 4 * (lane >> 4) + i;
      if ((lane & 15) == 0 && tile_ok[k] && row < dm.rows)
        partial[((int64_t)lg * nchunk + ck) * dm.rows + row] = make_float4(mV[k][i], zV[k][i], mC[k][i], zC[k][i]);
    }
  }
}

// K5b: merge chunk partials in order; S = sum_r exp(m_C - m_V) Z_C / Z_V.
__global__ __launch_bounds__(256) void k_rowstats_combine(Dims dm, const float4* __restrict__ partial, int nchunk,
                                                          TreeView tv) {
  const int lg = blockIdx.x;
  __shared__ float red[256];
  float acc = 0.f;
  for (int r = threadIdx.x; r < dm.rows; r += 256) {
    float mv = -INFINITY, zv = 0.f, mc = -INFINITY, zc = 0.f;
    for (int c = 0; c < nchunk; ++c) {
      float4 p = partial[((int64_t)lg * nchunk + c) * dm.rows + r];
      lse_merge(mv, zv, p.x, p.y);
      lse_merge(mc, zc, p.z, p.w);
    }
    tv.row_stats[(int64_t)lg * dm.rows + r] = make_float4(mv, zv, mc, zc);
    if (zc > 0.f) acc += expf(mc - mv) * zc / zv;
    const int u = r % dm.W, hl = r / dm.W;
    if (u % dm.hpg == hl) {                    // row of distortion probe u (round-robin heads)
      tv.probe_m[(int64_t)lg * dm.W + u] = mc;
      tv.probe_ZC[(int64_t)lg * dm.W + u] = zc;
    }
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) tv.lg_S[lg] = red[0];
}

hipError_t launch_rowstats(const Dims& dm, const void* K, const void* Q, const TreeView& tv, float4* partial,
                           hipStream_t st) {
  const int nchunk = rowstats_chunks(dm);
  dim3 grid(nchunk, dm.L * dm.G, (dm.rows + 255) / 256);
  if (dm.dtype == GRACEKV_BF16) {
    if (dm.d == 128)
      hipLaunchKernelGGL((k_rowstats<uint16_t, 128>), grid, dim3(256), 0, st, dm, (const uint16_t*)K, (const uint16_t*)Q, partial, nchunk);
    else
      hipLaunchKernelGGL((k_rowstats<uint16_t, 64>), grid, dim3(256), 0, st, dm, (const uint16_t*)K, (const uint16_t*)Q, partial, nchunk);
  } else {
    if (dm.d == 128)
      hipLaunchKernelGGL((k_rowstats<float, 128>), grid, dim3(256), 0, st, dm, (const float*)K, (const float*)Q, partial, nchunk);
    else
      hipLaunchKernelGGL((k_rowstats<float, 64>), grid, dim3(256), 0, st, dm, (const float*)K, (const float*)Q, partial, nchunk);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_rowstats_combine, dim3(dm.L * dm.G), dim3(256), 0, st, dm, (const float4*)partial, nchunk, tv);
  return hipGetLastError();
}

// ---- MFMA layout self-test --------------------------------------------------
__global__ void k_selftest_mfma(int which, float* out) {
  const int lane = threadIdx.x;
  // A[i][k] = (i - 3k) / 8, B[j][k] = (2j + k) / 16 -- exact in bf16 for 0 <= i, j, k < 16
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  if (which == 1) {
    s16x4 a, b;
    for (int q = 0; q < 4; ++q) {
      int k = 4 * (lane >> 4) + q;
      a[q] = (short)f32_to_bf16_rne((float)((lane & 15) - 3 * k) / 8.f);
      b[q] = (short)f32_to_bf16_rne((float)(2 * (lane & 15) + k) / 16.f);
    }
    acc = mfma_bf16_16x16x16(a, b, acc);
  } else {
    for (int s = 0; s < 4; ++s) {
      int k = 4 * s + (lane >> 4);
      acc = mfma_f32_16x16x4((float)((lane & 15) - 3 * k) / 8.f, (float)(2 * (lane & 15) + k) / 16.f, acc);
    }
  }
  for (int r = 0; r < 4; ++r) out[(4 * (lane >> 4) + r) * 16 + (lane & 15)] = acc[r];
}

hipError_t selftest_mfma(int which, float* host_out) {
  float* d = nullptr;
  hipError_t e = hipMalloc(&d, 256 * sizeof(float));
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_selftest_mfma, dim3(1), dim3(64), 0, 0, which, d);
  e = hipGetLastError();
  if (e == hipSuccess) e = hipMemcpy(host_out, d, 256 * sizeof(float), hipMemcpyDeviceToHost);
  hipFree(d);
  return e;
}

}  // namespace gkv
