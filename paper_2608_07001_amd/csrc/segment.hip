// Curvature-guided slot segmentation (App. B.2 - B.3).
//
// K1  seg_curvature: per slab and 64-position tile, L2-normalised hidden rows
//     (eq:app_hidden_normalization; norms from the Gram diagonal of K3) are
//     staged in LDS column-chunk by column-chunk; each position accumulates, for w in {4, 8, 16}, the three
//     dot products of delta_- = hbar_i - mean(hbar_{i-w+1..i}) and
//     delta_+ = mean(hbar_{i+1..i+w}) - hbar_i (eq:app_local_means,
//     eq:app_local_directions), giving kappa^{(l,w)} (eq:app_local_curvature;
//     zero outside w <= i < T - w), and ||hbar_{i+1} - hbar_i||^2 for the
//     dispersion (eq:app_adjacent_difference).
// K1b seg_stabilize: kappa_i = Mean - lam_stab * population Std over the
//     |L_seg| x 3 values (eq:app_stabilized_curvature).
// K2  seg_robust_z: lower medians by radix select on order-preserving keys;
//     b_i = z(kappa_i) + lam_s z(s_i) (eq:app_robust_z, eq:app_mad,
//     eq:app_boundary_score).
// K3  seg_gram: banded Gram <h_i, h_j>, 0 <= i - j < 128, of the raw hidden
//     rows with MFMA (bf16 products are exact), LDS-tiled for bf16.  Since the prefix sums of d_t
//     telescope, sum_{t=a}^{e-2} d_t = hbar_{e-1} - hbar_a, and
//     ||hbar_i - hbar_j||^2 follows from the Gram and the row norms; with the
//     fp64 prefix of ||d_t||^2 this gives the dispersion in O(1) per slot
//     (eq:app_prefix_dispersion, eq:app_slot_dispersion).
// K4  seg_dp: slot scores tabulated in parallel (fp64), then the DP of
//     eq:app_dp_recurrence by one workgroup.  With n_min >= 16, F[i .. i+15]
//     depend only on F[< i], so 16 ends advance per step; ties go to the
//     smallest predecessor; terminal relaxation eq:app_terminal_predecessor;
//     backtrack from LDS.
#include "common.h"

namespace gkv {

constexpr int CT = 64;                  // positions per curvature tile (one per lane)
constexpr int CHALO = 16;               // max window
constexpr int CROWS = CT + 2 * CHALO;   // rows staged (i0 - 16 .. i0 + 80)
constexpr int CCOL = 64;                // columns per LDS chunk
constexpr int CLD = CCOL + 4;           // LDS row stride: 16-byte reads of 16 consecutive rows hit distinct banks
constexpr int BAND = 128;

struct SegWs {
  float* kap9;      // [n_seg * 3][T]
  float* sqd;       // [n_seg][T]
  float* sq;        // [T]
  float* gram;      // [n_seg][T][BAND]
  float* dist2;     // [N_c][BAND]
  double* P2;       // [N_c + 1]
  uint8_t* Poff;    // [N_c + 1]
  float* scratch;   // [T] for the robust z
  double* Fdbg;     // [1]
  double* S;        // [N_c][128] slot scores by (i, length), candidate-major per lane
};

static size_t al(size_t x) { return (x + 255) & ~(size_t)255; }

size_t segment_ws_bytes(const Dims& dm) {
  const size_t T = (size_t)dm.T, N = (size_t)dm.N_c;
  return al(dm.n_seg * 3 * T * 4) + al(dm.n_seg * T * 4) + al(T * 4) + al((size_t)dm.n_seg * T * BAND * 4) +
         al(N * BAND * 4) + al((N + 1) * 8) + al(N + 1) + al(T * 4) + al(8) + al(N * BAND * 8);
}

static SegWs seg_view(void* ws, const Dims& dm) {
  const size_t T = (size_t)dm.T, N = (size_t)dm.N_c;
  char* p = (char*)ws;
  SegWs s;
  s.kap9 = (float*)p; p += al(dm.n_seg * 3 * T * 4);
  s.sqd = (float*)p; p += al(dm.n_seg * T * 4);
  s.sq = (float*)p; p += al(T * 4);
  s.gram = (float*)p; p += al((size_t)dm.n_seg * T * BAND * 4);
  s.dist2 = (float*)p; p += al(N * BAND * 4);
  s.P2 = (double*)p; p += al((N + 1) * 8);
  s.Poff = (uint8_t*)p; p += al(N + 1);
  s.scratch = (float*)p; p += al(T * 4);
  s.Fdbg = (double*)p; p += al(8);
  s.S = (double*)p;
  return s;
}

// Lane p owns position i0 + p; wave w owns the column quads w, w + 4, ... of
// each 64-column chunk and keeps partial dot products, summed over the waves
// at the end.  Rows are scaled by 1 / max(||h||, eps) while staged, the norm
// taken from the diagonal of the banded Gram (computed first).
template <typename T>
__global__ __launch_bounds__(256) void k_curvature(Dims dm, const T* __restrict__ hidden, SegWs ws) {
  __shared__ float inv[CROWS];
  __shared__ __align__(16) float hb[CROWS * CLD];
  __shared__ float red[4][10][CT];
  const int slab = blockIdx.y;
  const int64_t i0 = (int64_t)blockIdx.x * CT;
  const int64_t T_ = dm.T;
  const int Dh = dm.Dh;
  const T* H = hidden + (int64_t)slab * T_ * Dh;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  if (tid < CROWS) {
    const int64_t i = i0 - CHALO + tid;
    float v = 0.f;
    if (i >= 0 && i < T_) v = 1.0f / fmaxf(sqrtf(ws.gram[((int64_t)slab * T_ + i) * BAND]), dm.eps_seg);
    inv[tid] = v;
  }
  const int rr = lane + CHALO;
  float acc[3][3], accD = 0.f;
#pragma unroll
  for (int w = 0; w < 3; ++w) acc[w][0] = acc[w][1] = acc[w][2] = 0.f;
  constexpr int EPL = 16 / (int)sizeof(T);          // elements per 16-byte load
  constexpr int LPR = CCOL / EPL;                   // loads per staged row
  for (int c0 = 0; c0 < Dh; c0 += CCOL) {
    __syncthreads();
    for (int e = tid; e < CROWS * LPR; e += 256) {
      const int r = e / LPR, c = (e % LPR) * EPL;
      const int64_t i = i0 - CHALO + r;
      float x[EPL];
#pragma unroll
      for (int k = 0; k < EPL; ++k) x[k] = 0.f;
      if (i >= 0 && i < T_ && c0 + c < Dh) {
        const float sc = inv[r];
        if constexpr (sizeof(T) == 2) {
          const uint4 u = *(const uint4*)(H + i * Dh + c0 + c);
          const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
          for (int h = 0; h < 4; ++h) {
            x[2 * h] = __uint_as_float(w4[h] << 16) * sc;
            x[2 * h + 1] = __uint_as_float(w4[h] & 0xffff0000u) * sc;
          }
        } else {
          const float4 u = *(const float4*)((const float*)H + i * Dh + c0 + c);
          x[0] = u.x * sc; x[1] = u.y * sc; x[2] = u.z * sc; x[3] = u.w * sc;
        }
      }
#pragma unroll
      for (int k = 0; k < EPL; k += 4) *(float4*)(hb + r * CLD + c + k) = make_float4(x[k], x[k + 1], x[k + 2], x[k + 3]);
    }
    __syncthreads();
#pragma unroll 1
    for (int qd = wave; qd < CCOL / 4; qd += 4) {
      const int c = 4 * qd;
      const float4 x4 = *(const float4*)(hb + rr * CLD + c);
      const float xv[4] = {x4.x, x4.y, x4.z, x4.w};
      float sm[4] = {0.f, 0.f, 0.f, 0.f}, sp[4] = {0.f, 0.f, 0.f, 0.f};
      int tau = 0;
#pragma unroll
      for (int w = 0; w < 3; ++w) {
        const int ww = w == 0 ? 4 : (w == 1 ? 8 : 16);
#pragma unroll
        for (; tau < ww; ++tau) {
          const float4 a = *(const float4*)(hb + (rr - tau) * CLD + c);
          const float4 b = *(const float4*)(hb + (rr + 1 + tau) * CLD + c);
          sm[0] += a.x; sm[1] += a.y; sm[2] += a.z; sm[3] += a.w;
          sp[0] += b.x; sp[1] += b.y; sp[2] += b.z; sp[3] += b.w;
        }
        const float iw = 1.0f / (float)ww;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const float dmn = xv[k] - sm[k] * iw;
          const float dpl = sp[k] * iw - xv[k];
          acc[w][0] += dmn * dpl;
          acc[w][1] += dmn * dmn;
          acc[w][2] += dpl * dpl;
        }
      }
      const float4 n4 = *(const float4*)(hb + (rr + 1) * CLD + c);
      const float nv[4] = {n4.x, n4.y, n4.z, n4.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) { const float dd = nv[k] - xv[k]; accD += dd * dd; }
    }
  }
#pragma unroll
  for (int w = 0; w < 3; ++w)
#pragma unroll
    for (int k = 0; k < 3; ++k) red[wave][3 * w + k][lane] = acc[w][k];
  red[wave][9][lane] = accD;
  __syncthreads();
  if (wave == 0) {
    float v[10];
#pragma unroll
    for (int k = 0; k < 10; ++k) v[k] = red[0][k][lane] + red[1][k][lane] + red[2][k][lane] + red[3][k][lane];
    const int64_t i = i0 + lane;
    if (i < T_) {
#pragma unroll
      for (int w = 0; w < 3; ++w) {
        const int ww = dm.win[w];
        float kap = 0.f;
        if (i >= ww && i < T_ - ww) {
          const float nm = fmaxf(sqrtf(v[3 * w + 1]), dm.eps_seg), np = fmaxf(sqrtf(v[3 * w + 2]), dm.eps_seg);
          kap = 1.f - v[3 * w] / (nm * np);
        }
        ws.kap9[((int64_t)slab * 3 + w) * T_ + i] = kap;
      }
      ws.sqd[(int64_t)slab * T_ + i] = (i + 1 < T_) ? v[9] : 0.f;
    }
  }
}

__global__ void k_stabilize(Dims dm, SegWs ws, float* kappa) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= dm.T) return;
  const int nv = dm.n_seg * 3;
  float m = 0.f;
  for (int k = 0; k < nv; ++k) m += ws.kap9[(int64_t)k * dm.T + i];
  m /= (float)nv;
  float v = 0.f;
  for (int k = 0; k < nv; ++k) { const float d = ws.kap9[(int64_t)k * dm.T + i] - m; v += d * d; }
  kappa[i] = m - dm.lam_stab * sqrtf(v / (float)nv);
  float s = 0.f;
  for (int k = 0; k < dm.n_seg; ++k) s += ws.sqd[(int64_t)k * dm.T + i];
  ws.sq[i] = s / (float)dm.n_seg;
}

// ---- K2: robust z ---------------------------------------------------------
__device__ __forceinline__ uint32_t okey(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float okey_inv(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// value of rank `rank` (ascending, 0-based) of f(src[i]) = |src[i] - center| or src[i]
__device__ float block_select(const float* src, int64_t n, int64_t rank, bool absdev, float center, uint32_t* hist) {
  uint32_t prefix = 0;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    for (int k = threadIdx.x; k < 256; k += blockDim.x) hist[k] = 0;
    __syncthreads();
    for (int64_t i = threadIdx.x; i < n; i += blockDim.x) {
      const float v = absdev ? fabsf(src[i] - center) : src[i];
      const uint32_t k = okey(v);
      if (pass > 0 && (k >> (shift + 8)) != (prefix >> (shift + 8))) continue;
      atomicAdd(&hist[(k >> shift) & 255u], 1u);
    }
    __syncthreads();
    __shared__ uint32_t pick;
    __shared__ int64_t below;
    if (threadIdx.x == 0) {
      int64_t cum = 0;
      for (int k = 0; k < 256; ++k) {
        if (cum + hist[k] > rank) { pick = (uint32_t)k; below = cum; break; }
        cum += hist[k];
      }
    }
    __syncthreads();
    prefix |= pick << shift;
    rank -= below;
    __syncthreads();
  }
  return okey_inv(prefix);
}

__global__ __launch_bounds__(1024) void k_robust_z(Dims dm, const float* __restrict__ kappa,
                                                   const float* __restrict__ surp, float* bscore) {
  __shared__ uint32_t hist[256];
  const int64_t n = dm.T;
  const int64_t rk = (n - 1) / 2;
  const float mk = block_select(kappa, n, rk, false, 0.f, hist);
  const float madk = block_select(kappa, n, rk, true, mk, hist);
  const float ms = block_select(surp, n, rk, false, 0.f, hist);
  const float mads = block_select(surp, n, rk, true, ms, hist);
  const float dk = dm.mad * madk + dm.eps_seg, ds = dm.mad * mads + dm.eps_seg;
  for (int64_t i = threadIdx.x; i < n; i += blockDim.x)
    bscore[i] = (kappa[i] - mk) / dk + dm.lam_s * ((surp[i] - ms) / ds);
}

// ---- K3: banded Gram --------------------------------------------------------
// bf16: a workgroup owns 64 rows i0 .. i0+63 of one slab and the 192 rows
// j in [i0 - 128, i0 + 64) they pair with; 64-dim chunks of those rows are
// staged in LDS (double-buffered, 16-byte loads) and wave w accumulates the
// 16 x 16 tiles (i-tile w, j-tile w .. w + 8) that touch the band.  A lane
// supplies 16 consecutive dims of a chunk per operand (4 k-steps), so each
// operand is two 16-byte LDS reads.
constexpr int GB_I = 64;                 // rows i per workgroup
constexpr int GB_J = GB_I + BAND;        // rows j staged
constexpr int GB_C = 64;                 // dims per chunk
constexpr int GB_LD = GB_C + 8;          // LDS row stride (bf16)

__global__ __launch_bounds__(256) void k_gram_bf16(Dims dm, const uint16_t* __restrict__ hidden, SegWs ws) {
  __shared__ __align__(16) uint16_t sh[2][GB_J * GB_LD];
  const int slab = blockIdx.y;
  const int64_t i0 = (int64_t)blockIdx.x * GB_I;
  const int64_t j0 = i0 - BAND;
  const int64_t T_ = dm.T;
  const int Dh = dm.Dh;
  const uint16_t* H = hidden + (int64_t)slab * T_ * Dh;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, i16 = lane & 15, g4 = lane >> 4;
  f32x4 acc[9];
#pragma unroll
  for (int k = 0; k < 9; ++k) acc[k] = f32x4{0.f, 0.f, 0.f, 0.f};
  constexpr int CPR = GB_C / 8;          // 16-byte chunks per staged row
  auto stage = [&](int buf, int c0, uint4* reg) {
#pragma unroll
    for (int k = 0; k < (GB_J * CPR) / 256; ++k) {
      const int e = tid + 256 * k;
      const int r = e / CPR, c = (e % CPR) * 8;
      const int64_t row = j0 + r;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (row >= 0 && row < T_ && c0 + c < Dh) v = *(const uint4*)(H + row * Dh + c0 + c);
      reg[k] = v;
    }
  };
  auto store = [&](int buf, const uint4* reg) {
#pragma unroll
    for (int k = 0; k < (GB_J * CPR) / 256; ++k) {
      const int e = tid + 256 * k;
      const int r = e / CPR, c = (e % CPR) * 8;
      *(uint4*)(sh[buf] + r * GB_LD + c) = reg[k];
    }
  };
  uint4 reg[(GB_J * CPR) / 256];
  stage(0, 0, reg);
  store(0, reg);
  int buf = 0;
  for (int c0 = 0; c0 < Dh; c0 += GB_C) {
    __syncthreads();
    const bool more = c0 + GB_C < Dh;
    if (more) stage(buf ^ 1, c0 + GB_C, reg);              // next chunk in flight
    const uint16_t* base = sh[buf];
    // A: rows i0 + 16 w + i16 = staged row 128 + 16 w + i16
    const uint4* pa = (const uint4*)(base + (BAND + 16 * wave + i16) * GB_LD + 16 * g4);
    const uint4 a0 = pa[0], a1 = pa[1];
    const uint32_t aw[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
#pragma unroll
    for (int k = 0; k < 9; ++k) {
      const uint4* pb = (const uint4*)(base + (16 * (wave + k) + i16) * GB_LD + 16 * g4);
      const uint4 b0 = pb[0], b1 = pb[1];
      const uint32_t bw[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
#pragma unroll
      for (int s = 0; s < 4; ++s)
        acc[k] = mfma_bf16_16x16x16(pk4(aw[2 * s], aw[2 * s + 1]), pk4(bw[2 * s], bw[2 * s + 1]), acc[k]);
    }
    if (more) store(buf ^ 1, reg);
    buf ^= 1;
  }
  // C[i][j]: lane holds i = 4 g4 + r of the i-tile, j = i16 of the j-tile
#pragma unroll
  for (int k = 0; k < 9; ++k) {
    const int64_t j = j0 + 16 * (wave + k) + i16;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t i = i0 + 16 * wave + 4 * g4 + r;
      const int64_t dlt = i - j;
      if (i < T_ && j >= 0 && dlt >= 0 && dlt < BAND)
        ws.gram[((int64_t)slab * T_ + i) * BAND + dlt] = acc[k][r];
    }
  }
}

// fp32: one 16-row tile per workgroup, operands straight from memory
__global__ __launch_bounds__(192) void k_gram_f32(Dims dm, const float* __restrict__ hidden, SegWs ws) {
  const int slab = blockIdx.y;
  const int64_t i0 = (int64_t)blockIdx.x * 16;
  const int64_t T_ = dm.T;
  const int Dh = dm.Dh;
  const float* H = hidden + (int64_t)slab * T_ * Dh;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t ri = i0 + (lane & 15);
  const bool iok = ri < T_;
  f32x4 acc[3];
  int64_t rj[3];
  bool jok[3];
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    acc[k] = f32x4{0.f, 0.f, 0.f, 0.f};
    rj[k] = i0 - BAND + 16 * (wave * 3 + k) + (lane & 15);
    jok[k] = rj[k] >= 0 && rj[k] < T_;
  }
  for (int s = 0; s < Dh; s += 4) {
    const int kc = s + (lane >> 4);
    const float a = iok ? H[ri * Dh + kc] : 0.f;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      const float b = jok[k] ? H[rj[k] * Dh + kc] : 0.f;
      acc[k] = mfma_f32_16x16x4(a, b, acc[k]);
    }
  }
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const int64_t j = i0 - BAND + 16 * (wave * 3 + k) + (lane & 15);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t i = i0 + 4 * (lane >> 4) + r;
      const int64_t dlt = i - j;
      if (i < T_ && j >= 0 && dlt >= 0 && dlt < BAND)
        ws.gram[((int64_t)slab * T_ + i) * BAND + dlt] = acc[k][r];
    }
  }
}

// dist2[e][delta] = mean over slabs of ||hbar_e - hbar_{e-delta}||^2, e < N_c
__global__ void k_dist2(Dims dm, SegWs ws) {
  const int64_t e = blockIdx.x;
  const int dlt = threadIdx.x;
  const int64_t j = e - dlt;
  float acc = 0.f;
  if (dlt > 0 && j >= 0) {
    for (int s = 0; s < dm.n_seg; ++s) {
      const float* G = ws.gram + (int64_t)s * dm.T * BAND;
      const float gii = G[e * BAND], gjj = G[j * BAND], gij = G[e * BAND + dlt];
      const float ni = fmaxf(sqrtf(gii), dm.eps_seg), nj = fmaxf(sqrtf(gjj), dm.eps_seg);
      acc += gii / (ni * ni) + gjj / (nj * nj) - 2.f * gij / (ni * nj);
    }
    acc /= (float)dm.n_seg;
  }
  ws.dist2[e * BAND + dlt] = acc;
}

// P2[t] = sum_{tau < t} sq[tau] (fp64), t = 0..N_c
__global__ __launch_bounds__(1024) void k_prefix_sq(Dims dm, SegWs ws) {
  __shared__ double part[1024];
  __shared__ double carry;
  const int64_t N = dm.N_c;
  if (threadIdx.x == 0) { carry = 0.0; ws.P2[0] = 0.0; }
  __syncthreads();
  for (int64_t t0 = 0; t0 < N; t0 += 1024) {
    const int64_t t = t0 + threadIdx.x;
    const double v = (t < N - 1) ? (double)ws.sq[t] : 0.0;     // d_t exists for t <= N - 2
    part[threadIdx.x] = v;
    __syncthreads();
    for (int o = 1; o < 1024; o <<= 1) {
      const double x = threadIdx.x >= o ? part[threadIdx.x - o] : 0.0;
      __syncthreads();
      part[threadIdx.x] += x;
      __syncthreads();
    }
    if (t < N) ws.P2[t + 1] = carry + part[threadIdx.x];
    __syncthreads();
    if (threadIdx.x == 0) carry += part[1023];
    __syncthreads();
  }
}

// ---- K4: DP -----------------------------------------------------------------
// The slot score Gamma(a) - lam_d Disp([a, i)) - lam_n ((i - a - n0) / n0)^2 of
// eq:app_dp_recurrence does not depend on F: it is tabulated for every end i
// and length in parallel (fp64), then the recurrence only adds F[a] and takes
// the maximum.  Candidate c = len - n_min of end i is stored at
// S[(i - 1) * 128 + (c % 16) * 8 + c / 16], so the lane that owns candidates
// c = sub, sub + 16, ... reads 8 consecutive doubles.
__device__ __forceinline__ void dp_better(double& bv, int64_t& ba, double v, int64_t a) {
  if (v > bv || (v == bv && a < ba)) { bv = v; ba = a; }
}

__device__ __forceinline__ void dp_better32(double& bv, int& ba, double v, int a) {
  if (v > bv || (v == bv && a < ba)) { bv = v; ba = a; }
}
// one DPP step of the (value, smallest start) maximum within 16-lane rows
// (an absent candidate is (-inf, INT_MAX) and never wins)
template <int CTRL>
__device__ __forceinline__ void dp_step(double& bv, int& ba) {
  const long long b = __double_as_longlong(bv);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(b & 0xffffffffll), CTRL, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(b >> 32), CTRL, 0xf, 0xf, false);
  const int a2 = __builtin_amdgcn_update_dpp(0, ba, CTRL, 0xf, 0xf, false);
  const double v2 = __longlong_as_double(((long long)hi << 32) | (long long)(unsigned)lo);
  const bool better = v2 > bv || (v2 == bv && a2 < ba);
  bv = better ? v2 : bv;
  ba = better ? a2 : ba;
}
// every lane of a 16-lane row ends with the row's best: lanes ^1, ^2 (quad
// permutes), then rotations by 4 and 8 within the row
__device__ __forceinline__ void dp_reduce16(double& bv, int& ba) {
  dp_step<0xB1>(bv, ba);     // quad_perm(1, 0, 3, 2)
  dp_step<0x4E>(bv, ba);     // quad_perm(2, 3, 0, 1)
  dp_step<0x124>(bv, ba);    // row_ror:4
  dp_step<0x128>(bv, ba);    // row_ror:8
}

__device__ __forceinline__ double slot_score(const Dims& dm, const float* __restrict__ b, const SegWs& ws, int64_t i,
                                             int len) {
  const int64_t a = i - len;
  const double gam = a == 0 ? 0.0 : (double)b[a - 1] - (double)dm.c_cut;
  const int nS = len - 1;
  double disp = 0.0;
  if (nS >= 1) {
    const double s2 = ws.P2[i - 1] - ws.P2[a];
    const double dd = (double)ws.dist2[(i - 1) * BAND + (len - 1)];
    disp = (s2 - dd / nS) / (double)(nS - 1 > 1 ? nS - 1 : 1);
  }
  const double x = (len - (double)dm.n0) / (double)dm.n0;
  return gam - (double)dm.lam_d * disp - (double)dm.lam_n * x * x;
}

__global__ __launch_bounds__(128) void k_slot_scores(Dims dm, const float* __restrict__ b, SegWs ws) {
  const int64_t i = (int64_t)blockIdx.x + 1;
  const int c = threadIdx.x;
  const int len = dm.n_min + c;
  double v = -INFINITY;
  if (len <= dm.n_max && i - len >= 0) v = slot_score(dm, b, ws, i, len);
  ws.S[(i - 1) * BAND + (c % 16) * 8 + c / 16] = v;
}

// F over [1, N] in steps of 16 ends (an end depends only on ends >= 16
// positions earlier): wave w owns ends i0 + 4 w .. i0 + 4 w + 3, 16 lanes per
// end, each lane 8 candidate lengths; ties go to the smallest start.  Terminal
// relaxation eq:app_terminal_predecessor, then the backtrack.
__global__ __launch_bounds__(256) void k_dp(Dims dm, const float* __restrict__ b, SegWs ws, int32_t* slots,
                                            int32_t* nslots, int use_lds) {
  extern __shared__ __align__(16) char dsm[];
  __shared__ double Fr[256];                 // F ring indexed by end & 255
  uint8_t* Poff = use_lds ? (uint8_t*)dsm : ws.Poff;
  const int64_t N = dm.N_c;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int st = lane >> 4, sub = lane & 15;
  if (N <= 0) {
    if (tid == 0) { slots[0] = 0; *nslots = 0; }
    return;
  }
  Fr[tid] = -INFINITY;
  __syncthreads();
  if (tid == 0) { Fr[0] = 0.0; Poff[0] = 0; }
  __syncthreads();
  // unconditional loads (row clamped to N) keep the load counter exact
  auto load = [&](int64_t i, double* sv) {
    const int64_t ic = i <= N ? i : N;
    const double2* p = (const double2*)(ws.S + (ic - 1) * BAND + sub * 8);
#pragma unroll
    for (int k = 0; k < 4; ++k) { const double2 v = p[k]; sv[2 * k] = v.x; sv[2 * k + 1] = v.y; }
  };
  // scores of 4 steps in flight (static register indices: the step loop is unrolled by 4)
  double sv[4][8];
#pragma unroll
  for (int q = 0; q < 4; ++q) load(1 + 16 * q + 4 * wave + st, sv[q]);
  for (int64_t i00 = 1; i00 <= N; i00 += 64) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t i0 = i00 + 16 * q;
      if (i0 > N) break;
      const int64_t i = i0 + 4 * wave + st;
      // all F reads first, then a branch-free (value, smallest start) maximum
      double Fa[8];
      int av[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int len = dm.n_min + sub + 16 * k;
        const int64_t a = i - len;
        const bool ok = i <= N && len <= dm.n_max && a >= 0;
        av[k] = ok ? (int)a : 0x7fffffff;
        Fa[k] = Fr[ok ? (int)(a & 255) : 0];
      }
      double bv = -INFINITY;
      int ba = 0x7fffffff;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const bool ok = av[k] != 0x7fffffff && Fa[k] != -INFINITY;
        const double v = ok ? Fa[k] + sv[q][k] : -INFINITY;
        const int a = ok ? av[k] : 0x7fffffff;
        const bool better = v > bv || (v == bv && a < ba);
        bv = better ? v : bv;
        ba = better ? a : ba;
      }
      load(i + 64, sv[q]);                   // the same lane's end four steps later
      dp_reduce16(bv, ba);
      lds_barrier();                         // every end of this step has read its F
      if (sub == 0 && i <= N) {
        Fr[i & 255] = bv;
        Poff[i] = ba != 0x7fffffff ? (uint8_t)(i - ba) : 0;
      }
      lds_barrier();                         // (Poff is only read after the loop's final full barrier)
    }
  }
  // terminal relaxation of the last slot's minimum length
  if (Poff[N] == 0 && wave == 0) {
    double bv = -INFINITY;
    int64_t ba = -1;
    for (int len = 1 + lane; len <= dm.n_max; len += 64) {
      const int64_t a = N - len;
      if (a < 0) continue;
      const double Fa = Fr[a & 255];
      if (Fa == -INFINITY) continue;
      dp_better(bv, ba, Fa + slot_score(dm, b, ws, N, len), a);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const double v2 = __shfl_xor(bv, o, 64);
      const int64_t a2 = __shfl_xor(ba, o, 64);
      if (a2 >= 0) dp_better(bv, ba, v2, a2);
    }
    if (lane == 0) { Poff[N] = ba >= 0 ? (uint8_t)(N - ba) : 0; ws.Fdbg[0] = bv; }
  } else if (tid == 0) {
    ws.Fdbg[0] = Fr[N & 255];
  }
  __syncthreads();
  if (tid == 0) {
    int J = 0;
    for (int64_t i = N; i > 0; i -= Poff[i]) {
      if (Poff[i] == 0) break;
      ++J;
    }
    int idx = J - 1;
    for (int64_t i = N; i > 0 && idx >= 0; i -= Poff[i]) slots[idx--] = (int32_t)(i - Poff[i]);
    slots[J] = (int32_t)N;
    *nslots = J;
  }
}

hipError_t launch_segment(const Dims& dm, const void* hidden, const float* surprisal, float* kappa, float* bscore,
                          int32_t* slot_starts, int32_t* n_slots, void* wsp, hipStream_t st) {
  SegWs ws = seg_view(wsp, dm);
  const dim3 g1((unsigned)((dm.T + CT - 1) / CT), dm.n_seg);
  // the Gram first: its diagonal gives the row norms of the curvature pass
  if (dm.dtype == GRACEKV_BF16) {
    const dim3 g3((unsigned)((dm.T + GB_I - 1) / GB_I), dm.n_seg);
    hipLaunchKernelGGL(k_gram_bf16, g3, dim3(256), 0, st, dm, (const uint16_t*)hidden, ws);
    hipLaunchKernelGGL(k_curvature<uint16_t>, g1, dim3(256), 0, st, dm, (const uint16_t*)hidden, ws);
  } else {
    const dim3 g3((unsigned)((dm.T + 15) / 16), dm.n_seg);
    hipLaunchKernelGGL(k_gram_f32, g3, dim3(192), 0, st, dm, (const float*)hidden, ws);
    hipLaunchKernelGGL(k_curvature<float>, g1, dim3(256), 0, st, dm, (const float*)hidden, ws);
  }
  hipLaunchKernelGGL(k_stabilize, dim3((unsigned)((dm.T + 255) / 256)), dim3(256), 0, st, dm, ws, kappa);
  hipLaunchKernelGGL(k_robust_z, dim3(1), dim3(1024), 0, st, dm, (const float*)kappa, surprisal, bscore);
  if (dm.N_c > 0) {
    hipLaunchKernelGGL(k_dist2, dim3((unsigned)dm.N_c), dim3(BAND), 0, st, dm, ws);
    hipLaunchKernelGGL(k_prefix_sq, dim3(1), dim3(1024), 0, st, dm, ws);
  }
  const size_t lds = (size_t)dm.N_c + 1;
  const int use_lds = lds <= 150 * 1024 ? 1 : 0;
  const size_t dyn = use_lds ? ((lds + 15) & ~(size_t)15) : 0;
  if (dyn > 0) {
    hipError_t e = hipFuncSetAttribute((const void*)k_dp, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
    if (e != hipSuccess) return e;
  }
  if (dm.N_c > 0)
    hipLaunchKernelGGL(k_slot_scores, dim3((unsigned)dm.N_c), dim3(BAND), 0, st, dm, (const float*)bscore, ws);
  hipLaunchKernelGGL(k_dp, dim3(1), dim3(256), dyn, st, dm, (const float*)bscore, ws, slot_starts, n_slots, use_lds);
  return hipGetLastError();
}

}  // namespace gkv
