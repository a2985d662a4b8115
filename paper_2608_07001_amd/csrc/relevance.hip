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
// Pass 1: grid (chunks of T, L*G, row groups of 256).  Each workgroup stages
// 64-token sub-chunks of K in LDS (16-byte loads, the next sub-chunk in flight
// while the current one is used) and forms transposed 16x16 logit tiles on the
// matrix cores (tokens x rows, 16x16x32 steps for bf16; exact products, fp32
// accumulation), so each lane holds 4 tokens of one row.  A
// token t < N_c is in both C and V(u); the lane keeps one online (max,
// sum-exp) pair over C and one over the visible tail [N_c, N_ctx + u], merged
// into V afterwards.  Pass 2 (combine): per (l, g), merge the chunk partials
// in order and reduce S.
#include "common.h"

namespace gkv {

constexpr int RS_SUB = 64;      // tokens per LDS sub-chunk
constexpr int RS_CHUNK = 2048;  // tokens per workgroup

int rowstats_chunks(const Dims& dm) { return (int)((dm.T + RS_CHUNK - 1) / RS_CHUNK); }

// online (max, sum-exp) update with four values (-inf = absent)
__device__ __forceinline__ void lse_add4(float& m, float& z, float x0, float x1, float x2, float x3) {
  const float mn = fmaxf(m, fmaxf(fmaxf(x0, x1), fmaxf(x2, x3)));
  if (mn == -INFINITY) return;
  if (mn > m) z *= fexp(m - mn);
  z += fexp(x0 - mn) + fexp(x1 - mn) + fexp(x2 - mn) + fexp(x3 - mn);
  m = mn;
}

template <typename T, int D>
__global__ __launch_bounds__(256) void k_rowstats(Dims dm, const T* __restrict__ K, const T* __restrict__ Q,
                                                  float4* __restrict__ partial, int nchunk) {
  constexpr bool BF = sizeof(T) == 2;
  constexpr int QE = D / 4;                       // elements of a lane's quarter row
  constexpr int QW = BF ? QE / 2 : QE;            // ... in 32-bit words
  constexpr int LDK = BF ? D + 8 : D + 4;
  constexpr int CH = 16 / (int)sizeof(T);         // elements per 16-byte chunk
  __shared__ __align__(16) T sK[RS_SUB * LDK];

  const int ck = blockIdx.x, lg = blockIdx.y, rg = blockIdx.z;
  const int l = lg / dm.G, g = lg % dm.G;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, i16 = lane & 15, g4 = lane >> 4;
  const int64_t t_begin = (int64_t)ck * RS_CHUNK;
  const int64_t t_end = min(dm.T, t_begin + RS_CHUNK);
  const T* Kp = K + (int64_t)lg * dm.T * D;
  const T* Qp = Q + ((int64_t)l * dm.H + (int64_t)g * dm.hpg) * dm.W * D;
  const float scale = 1.0f / sqrtf((float)D);

  // the wave's 4 row tiles: Q quarter rows in registers
  uint32_t qreg[4][QW];
  int vlim[4];                    // last visible position N_ctx + u of the lane's row
  bool tile_ok[4], rok[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int rt = rg * 16 + wave * 4 + k;
    tile_ok[k] = rt * 16 < dm.rows;
    const int row = rt * 16 + i16;
    rok[k] = row < dm.rows;
    vlim[k] = (int)dm.N_ctx + (rok[k] ? row % dm.W : 0);
    const uint4* q4 = (const uint4*)(Qp + (int64_t)(rok[k] ? row : 0) * D + QE * g4);
#pragma unroll
    for (int h = 0; h < QW / 4; ++h) {
      const uint4 v = q4[h];
      qreg[k][4 * h] = v.x; qreg[k][4 * h + 1] = v.y; qreg[k][4 * h + 2] = v.z; qreg[k][4 * h + 3] = v.w;
    }
  }
  float mC[4], zC[4], mT[4], zT[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) { mC[k] = -INFINITY; zC[k] = 0.f; mT[k] = -INFINITY; zT[k] = 0.f; }

  // the next sub-chunk is loaded into registers while the current one is used
  constexpr int NLD = RS_SUB * (D / CH) / 256;    // 16-byte loads per thread per sub-chunk
  uint4 pre[NLD];
  auto load_sub = [&](int64_t s0) {
#pragma unroll
    for (int q = 0; q < NLD; ++q) {
      const int e = tid + 256 * q;
      const int tr = e / (D / CH), c = (e % (D / CH)) * CH;
      const int64_t t = s0 + tr;
      pre[q] = t < t_end ? *(const uint4*)(Kp + t * D + c) : make_uint4(0, 0, 0, 0);
    }
  };
  load_sub(t_begin);
  for (int64_t s0 = t_begin; s0 < t_end; s0 += RS_SUB) {
    __syncthreads();
#pragma unroll
    for (int q = 0; q < NLD; ++q) {              // stage K[s0 .. s0+SUB), zero past the chunk
      const int e = tid + 256 * q;
      const int tr = e / (D / CH), c = (e % (D / CH)) * CH;
      *(uint4*)(sK + tr * LDK + c) = pre[q];
    }
    if (s0 + RS_SUB < t_end) load_sub(s0 + RS_SUB);
    __syncthreads();
    const bool allC = s0 + RS_SUB <= dm.N_c && s0 + RS_SUB <= t_end;
#pragma unroll
    for (int tt = 0; tt < RS_SUB / 16; ++tt) {
      uint32_t kreg[QW];
      const uint4* k4 = (const uint4*)(sK + (tt * 16 + i16) * LDK + QE * g4);
#pragma unroll
      for (int h = 0; h < QW / 4; ++h) {
        const uint4 v = k4[h];
        kreg[4 * h] = v.x; kreg[4 * h + 1] = v.y; kreg[4 * h + 2] = v.z; kreg[4 * h + 3] = v.w;
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (!tile_ok[k]) continue;
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        if constexpr (BF) {
          // dims QE g4 + 8 s .. + 7 of the lane's token and row per 16x16x32 step
#pragma unroll
          for (int s = 0; s < QE / 8; ++s)
            acc = mfma_bf16_16x16x32(
                pk8(make_uint4(kreg[4 * s], kreg[4 * s + 1], kreg[4 * s + 2], kreg[4 * s + 3])),
                pk8(make_uint4(qreg[k][4 * s], qreg[k][4 * s + 1], qreg[k][4 * s + 2], qreg[k][4 * s + 3])), acc);
        } else {
#pragma unroll
          for (int s = 0; s < QE; ++s) acc = mfma_f32_16x16x4(__uint_as_float(kreg[s]), __uint_as_float(qreg[k][s]), acc);
        }
        // lane holds tokens s0 + 16 tt + 4 g4 + r of its row
        float x[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) x[r] = acc[r] * scale;
        if (allC) {
          if (rok[k]) lse_add4(mC[k], zC[k], x[0], x[1], x[2], x[3]);
        } else {
          float xc[4], xt[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int64_t t = s0 + 16 * tt + 4 * g4 + r;
            const bool vis = rok[k] && t < t_end && t <= vlim[k];
            const bool inC = vis && t < dm.N_c;
            xc[r] = inC ? x[r] : -INFINITY;
            xt[r] = (vis && !inC) ? x[r] : -INFINITY;
          }
          lse_add4(mC[k], zC[k], xc[0], xc[1], xc[2], xc[3]);
          lse_add4(mT[k], zT[k], xt[0], xt[1], xt[2], xt[3]);
        }
      }
    }
  }
  // merge the 4 lanes holding the same row (disjoint token subsets)
#pragma unroll
  for (int k = 0; k < 4; ++k) {
#pragma unroll
    for (int o = 16; o < 64; o <<= 1) {
      float m2 = __shfl_xor(mC[k], o, 64), z2 = __shfl_xor(zC[k], o, 64);
      lse_merge(mC[k], zC[k], m2, z2);
      m2 = __shfl_xor(mT[k], o, 64);
      z2 = __shfl_xor(zT[k], o, 64);
      lse_merge(mT[k], zT[k], m2, z2);
    }
    const int row = (rg * 16 + wave * 4 + k) * 16 + i16;
    if (g4 == 0 && tile_ok[k] && rok[k])
      partial[((int64_t)lg * nchunk + ck) * dm.rows + row] = make_float4(mC[k], zC[k], mT[k], zT[k]);
  }
}

// bf16 keys: 16x16x32 steps with the operands held as 16-byte register
// tuples (no repacking), two token tiles per statistics update, and the C
// statistics kept in base-2 units (logit * scale * log2 e) with a branch-free
// running maximum; converted to natural units at the end.
// Running (max, sum 2^(y - max)) update with eight values; -inf values are absent.
__device__ __forceinline__ void lse2_add8(float& m, float& z, const float* y) {
  const float mx = fmaxf(fmaxf(fmaxf(y[0], y[1]), fmaxf(y[2], y[3])), fmaxf(fmaxf(y[4], y[5]), fmaxf(y[6], y[7])));
  const float mn = fmaxf(m, mx);
  const float ms = mn == -INFINITY ? 0.f : mn;    // all absent so far: keep (−inf, 0)
  float acc = z * __builtin_amdgcn_exp2f(m - ms);
#pragma unroll
  for (int r = 0; r < 8; ++r) acc += __builtin_amdgcn_exp2f(y[r] - ms);
  z = acc;
  m = mn;
}

// The same update from eight raw logits x (y = x * sc2, sc2 > 0, all present):
// the maximum is taken on x (scaling by a positive number keeps the order, and
// rounding is monotonic, so max(x) * sc2 is the largest y), and each term is
// 2^(x * sc2 - max) with the product fused into the subtraction.
// The maximum is taken as med3(a, b, +inf), which equals max(a, b) for any
// a, b that are not NaN and, unlike fmaxf, needs no quieting of its operands;
// pinf holds +inf in a register the optimiser cannot see through (an empty asm
// statement, no instruction), so the median is not folded back into a maximum.
__device__ __forceinline__ float opaque_inf() {
  float v = INFINITY;
  asm volatile("" : "+v"(v));
  return v;
}
__device__ __forceinline__ void lse2_add8_raw(float& m, float& z, const float* x, float sc2, float pinf) {
  auto mx = [pinf](float a, float b) { return __builtin_amdgcn_fmed3f(a, b, pinf); };
  const float mxr = mx(mx(mx(x[0], x[1]), mx(x[2], x[3])), mx(mx(x[4], x[5]), mx(x[6], x[7])));
  const float mn = mx(m, mxr * sc2);
  float e[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) e[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(x[r], sc2, -mn));
  // pairwise: a short dependency chain instead of eight additions in a row
  const float s8 = ((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7]));
  z = __builtin_fmaf(z, __builtin_amdgcn_exp2f(m - mn), s8);   // m = -inf at first: 2^-inf = 0
  m = mn;
}

template <int D>
__global__ __launch_bounds__(256, 2) void k_rowstats_bf(Dims dm, const uint16_t* __restrict__ K,
                                                     const uint16_t* __restrict__ Q, float4* __restrict__ partial,
                                                     int nchunk) {
  constexpr int QE = D / 4;                       // elements of a lane's quarter row
  constexpr int KS = QE / 8;                      // 16x16x32 steps per tile
  constexpr int LDK = D + 8;
  constexpr int CH = 8;                           // elements per 16-byte chunk
  __shared__ __align__(16) uint16_t sK[RS_SUB * LDK];

  const int ck = blockIdx.x, lg = blockIdx.y, rg = blockIdx.z;
  const int l = lg / dm.G, g = lg % dm.G;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, i16 = lane & 15, g4 = lane >> 4;
  const int64_t t_begin = (int64_t)ck * RS_CHUNK;
  const int64_t t_end = min(dm.T, t_begin + RS_CHUNK);
  const uint16_t* Kp = K + (int64_t)lg * dm.T * D;
  const uint16_t* Qp = Q + ((int64_t)l * dm.H + (int64_t)g * dm.hpg) * dm.W * D;
  const float scale = 1.0f / sqrtf((float)D);
  const float sc2 = scale * 1.44269504088896341f;
  const float pinf = opaque_inf();

  // the wave's 4 row tiles: lane (row i16, group g4) holds dims QE g4 .. QE g4 + QE - 1
  uint4 qv[4][KS];
  int vlim[4];                    // last visible position N_ctx + u of the lane's row
  bool tile_ok[4], rok[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int rt = rg * 16 + wave * 4 + k;
    tile_ok[k] = rt * 16 < dm.rows;
    const int row = rt * 16 + i16;
    rok[k] = row < dm.rows;
    vlim[k] = (int)dm.N_ctx + (rok[k] ? row % dm.W : 0);
    const uint4* q4 = (const uint4*)(Qp + (int64_t)(rok[k] ? row : 0) * D + QE * g4);
#pragma unroll
    for (int s = 0; s < KS; ++s) qv[k][s] = q4[s];
  }
  float mC[4], zC[4], mT[4], zT[4];               // C in base-2 units, the tail in natural units
#pragma unroll
  for (int k = 0; k < 4; ++k) { mC[k] = -INFINITY; zC[k] = 0.f; mT[k] = -INFINITY; zT[k] = 0.f; }

  constexpr int NLD = RS_SUB * (D / CH) / 256;    // 16-byte loads per thread per sub-chunk
  uint4 pre[NLD];
  auto load_sub = [&](int64_t s0) {
#pragma unroll
    for (int q = 0; q < NLD; ++q) {
      const int e = tid + 256 * q;
      const int tr = e / (D / CH), c = (e % (D / CH)) * CH;
      const int64_t t = s0 + tr;
      pre[q] = t < t_end ? *(const uint4*)(Kp + t * D + c) : make_uint4(0, 0, 0, 0);
    }
  };
  load_sub(t_begin);
  for (int64_t s0 = t_begin; s0 < t_end; s0 += RS_SUB) {
    __syncthreads();
#pragma unroll
    for (int q = 0; q < NLD; ++q) {
      const int e = tid + 256 * q;
      const int tr = e / (D / CH), c = (e % (D / CH)) * CH;
      *(uint4*)(sK + tr * LDK + c) = pre[q];
    }
    if (s0 + RS_SUB < t_end) load_sub(s0 + RS_SUB);
    __syncthreads();
    const bool allC = s0 + RS_SUB <= dm.N_c && s0 + RS_SUB <= t_end;
    if (allC && tile_ok[3]) {
      // the common case, wave-uniform: every token of the block is in C and
      // visible to every window query, and the wave's four row tiles all
      // exist; one straight-line block per 32 tokens, so the products of one
      // tile overlap the exponentials of another (a lane of a row past the
      // last one computes on row 0's query; its statistics are never written)
#pragma unroll
      for (int tp = 0; tp < RS_SUB / 32; ++tp) {
        uint4 kv[2][KS];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const uint4* k4 = (const uint4*)(sK + (32 * tp + 16 * h + i16) * LDK + QE * g4);
#pragma unroll
          for (int s = 0; s < KS; ++s) kv[h][s] = k4[s];
        }
        f32x4 acc[4][2];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          acc[k][0] = f32x4{0.f, 0.f, 0.f, 0.f};
          acc[k][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int s = 0; s < KS; ++s)
#pragma unroll
            for (int h = 0; h < 2; ++h) acc[k][h] = mfma_bf16_16x16x32(pk8(kv[h][s]), pk8(qv[k][s]), acc[k][h]);
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          float y[8];
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int r = 0; r < 4; ++r) y[4 * h + r] = acc[k][h][r];
          lse2_add8_raw(mC[k], zC[k], y, sc2, pinf);
        }
      }
      continue;
    }
#pragma unroll
    for (int tp = 0; tp < RS_SUB / 32; ++tp) {
      uint4 kv[2][KS];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint4* k4 = (const uint4*)(sK + (32 * tp + 16 * h + i16) * LDK + QE * g4);
#pragma unroll
        for (int s = 0; s < KS; ++s) kv[h][s] = k4[s];
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (!tile_ok[k]) continue;
        f32x4 acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
          for (int h = 0; h < 2; ++h) acc[h] = mfma_bf16_16x16x32(pk8(kv[h][s]), pk8(qv[k][s]), acc[h]);
        // lane holds tokens s0 + 32 tp + 16 h + 4 g4 + r of its row
        float y[8];
        if (allC) {
          // every token of the block is in C and visible to every window query;
          // a lane of a row past the last one computes on row 0's query and its
          // statistics are never written
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int r = 0; r < 4; ++r) y[4 * h + r] = acc[h][r];
          lse2_add8_raw(mC[k], zC[k], y, sc2, pinf);
        } else {
          float xt[8];
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int64_t t = s0 + 32 * tp + 16 * h + 4 * g4 + r;
              const bool vis = rok[k] && t < t_end && t <= vlim[k];
              const bool inC = vis && t < dm.N_c;
              y[4 * h + r] = inC ? acc[h][r] * sc2 : -INFINITY;
              xt[4 * h + r] = (vis && !inC) ? acc[h][r] * scale : -INFINITY;
            }
          lse_add4(mT[k], zT[k], xt[0], xt[1], xt[2], xt[3]);
          lse_add4(mT[k], zT[k], xt[4], xt[5], xt[6], xt[7]);
          lse2_add8(mC[k], zC[k], y);
        }
      }
    }
  }
  // C statistics back to natural units; merge the 4 lanes holding the same row
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    mC[k] = mC[k] * 0.69314718055994531f;
#pragma unroll
    for (int o = 16; o < 64; o <<= 1) {
      float m2 = __shfl_xor(mC[k], o, 64), z2 = __shfl_xor(zC[k], o, 64);
      lse_merge(mC[k], zC[k], m2, z2);
      m2 = __shfl_xor(mT[k], o, 64);
      z2 = __shfl_xor(zT[k], o, 64);
      lse_merge(mT[k], zT[k], m2, z2);
    }
    const int row = (rg * 16 + wave * 4 + k) * 16 + i16;
    if (g4 == 0 && tile_ok[k] && rok[k])
      partial[((int64_t)lg * nchunk + ck) * dm.rows + row] = make_float4(mC[k], zC[k], mT[k], zT[k]);
  }
}

// K5b: merge chunk partials in order; S = sum_r exp(m_C - m_V) Z_C / Z_V.
__global__ __launch_bounds__(256) void k_rowstats_combine(Dims dm, const float4* __restrict__ partial, int nchunk,
                                                          TreeView tv) {
  const int lg = blockIdx.x;
  __shared__ float red[256];
  float acc = 0.f;
  for (int r = threadIdx.x; r < dm.rows; r += 256) {
    float mc = -INFINITY, zc = 0.f, mt = -INFINITY, zt = 0.f;
    for (int c = 0; c < nchunk; ++c) {
      const float4 p = partial[((int64_t)lg * nchunk + c) * dm.rows + r];
      lse_merge(mc, zc, p.x, p.y);
      lse_merge(mt, zt, p.z, p.w);
    }
    float mv = mc, zv = zc;                    // V(u) = C + the visible tail
    lse_merge(mv, zv, mt, zt);
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
      hipLaunchKernelGGL((k_rowstats_bf<128>), grid, dim3(256), 0, st, dm, (const uint16_t*)K, (const uint16_t*)Q, partial,
                         nchunk);
    else
      hipLaunchKernelGGL((k_rowstats_bf<64>), grid, dim3(256), 0, st, dm, (const uint16_t*)K, (const uint16_t*)Q, partial,
                         nchunk);
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
  if (which == 3) {                     // column sums over the four 16-lane rows
    out[lane] = col_sum4((float)(lane + 1));
    for (int i = 64 + lane; i < 256; i += 64) out[i] = 0.f;
    return;
  }
  if (which == 2) {                     // 16x16x32: k < 32
    s16x8 a, b;
    for (int q = 0; q < 8; ++q) {
      int k = 8 * (lane >> 4) + q;
      a[q] = (short)f32_to_bf16_rne((float)((lane & 15) - 3 * k) / 8.f);
      b[q] = (short)f32_to_bf16_rne((float)(2 * (lane & 15) + k) / 16.f);
    }
    acc = mfma_bf16_16x16x32(a, b, acc);
  } else if (which == 1) {
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

hipError_t selftest_mfma(int which, float* out, hipStream_t st) {
  hipLaunchKernelGGL(k_selftest_mfma, dim3(1), dim3(64), 0, st, which, out);
  return hipGetLastError();
}

}  // namespace gkv
