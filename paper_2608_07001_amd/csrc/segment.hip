// Curvature-guided slot segmentation (App. B.2 - B.3).
//
// K1  seg_curvature: per slab and 64-position tile, L2-normalised hidden rows
//     (eq:app_hidden_normalization) are staged in LDS column-chunk by
//     column-chunk; each position accumulates, for w in {4, 8, 16}, the three
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

constexpr int CT = 64;                  // positions per curvature tile
constexpr int CHALO = 16;               // max window
constexpr int CROWS = CT + 2 * CHALO;   // rows staged (i0 - 16 .. i0 + 80)
constexpr int CCOL = 64;                // columns per LDS chunk
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

template <typename T>
__global__ __launch_bounds__(256) void k_curvature(Dims dm, const T* __restrict__ hidden, SegWs ws) {
  __shared__ float nrm[CROWS];
  __shared__ float hb[CROWS][CCOL + 1];
  const int slab = blockIdx.y;
  const int64_t i0 = (int64_t)blockIdx.x * CT;
  const int64_t T_ = dm.T;
  const int Dh = dm.Dh;
  const T* H = hidden + (int64_t)slab * T_ * Dh;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  for (int rr = wave; rr < CROWS; rr += 4) {
    const int64_t i = i0 - CHALO + rr;
    float s = 0.f;
    if (i >= 0 && i < T_)
      for (int c = lane; c < Dh; c += 64) { const float x = ldf(H, i * Dh + c); s += x * x; }
    s = wave_sum(s);
    if (lane == 0) nrm[rr] = fmaxf(sqrtf(s), dm.eps_seg);
  }
  const int p = tid >> 2, qq = tid & 3;
  const int rr_i = p + CHALO;
  float acc[3][3], accD = 0.f;
#pragma unroll
  for (int w = 0; w < 3; ++w) acc[w][0] = acc[w][1] = acc[w][2] = 0.f;
  for (int c0 = 0; c0 < Dh; c0 += CCOL) {
    __syncthreads();
    for (int e = tid; e < CROWS * CCOL; e += 256) {
      const int rr = e / CCOL, c = e % CCOL;
      const int64_t i = i0 - CHALO + rr;
      float x = 0.f;
      if (i >= 0 && i < T_ && c0 + c < Dh) x = ldf(H, i * Dh + c0 + c) / nrm[rr];
      hb[rr][c] = x;
    }
    __syncthreads();
    for (int c = qq; c < CCOL; c += 4) {
      const float x = hb[rr_i][c];
      float sm = 0.f, sp = 0.f;
      int tau = 0;
#pragma unroll
      for (int w = 0; w < 3; ++w) {
        const int ww = w == 0 ? 4 : (w == 1 ? 8 : 16);
        for (; tau < ww; ++tau) {
          sm += hb[rr_i - tau][c];
          sp += hb[rr_i + 1 + tau][c];
        }
        const float dmn = x - sm / (float)ww;
        const float dpl = sp / (float)ww - x;
        acc[w][0] += dmn * dpl;
        acc[w][1] += dmn * dmn;
        acc[w][2] += dpl * dpl;
      }
      const float dd = hb[rr_i + 1][c] - x;
      accD += dd * dd;
    }
  }
#pragma unroll
  for (int w = 0; w < 3; ++w)
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      acc[w][k] += __shfl_xor(acc[w][k], 1, 64);
      acc[w][k] += __shfl_xor(acc[w][k], 2, 64);
    }
  accD += __shfl_xor(accD, 1, 64);
  accD += __shfl_xor(accD, 2, 64);
  const int64_t i = i0 + p;
  if (qq == 0 && i < T_) {
#pragma unroll
    for (int w = 0; w < 3; ++w) {
      const int ww = dm.win[w];
      float kap = 0.f;
      if (i >= ww && i < T_ - ww) {
        const float nm = fmaxf(sqrtf(acc[w][1]), dm.eps_seg), np = fmaxf(sqrtf(acc[w][2]), dm.eps_seg);
        kap = 1.f - acc[w][0] / (nm * np);
      }
      ws.kap9[((int64_t)slab * 3 + w) * T_ + i] = kap;
    }
    ws.sqd[(int64_t)slab * T_ + i] = (i + 1 < T_) ? accD : 0.f;
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
  auto load = [&](int64_t i, double* sv) {
    if (i <= N) {
      const double2* p = (const double2*)(ws.S + (i - 1) * BAND + sub * 8);
#pragma unroll
      for (int k = 0; k < 4; ++k) { const double2 v = p[k]; sv[2 * k] = v.x; sv[2 * k + 1] = v.y; }
    } else {
#pragma unroll
      for (int k = 0; k < 8; ++k) sv[k] = -INFINITY;
    }
  };
  double cur[8], nxt[8];
  load(1 + 4 * wave + st, cur);
  for (int64_t i0 = 1; i0 <= N; i0 += 16) {
    const int64_t i = i0 + 4 * wave + st;
    load(i + 16, nxt);                       // next step's scores in flight
    double bv = -INFINITY;
    int64_t ba = -1;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int len = dm.n_min + sub + 16 * k;
      const int64_t a = i - len;
      if (i <= N && len <= dm.n_max && a >= 0) {
        const double Fa = Fr[a & 255];
        if (Fa != -INFINITY) dp_better(bv, ba, Fa + cur[k], a);
      }
    }
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) {
      const double v2 = __shfl_xor(bv, o, 64);
      const int64_t a2 = __shfl_xor(ba, o, 64);
      if (a2 >= 0) dp_better(bv, ba, v2, a2);
    }
    __syncthreads();                         // every end of this step has read its F
    if (sub == 0 && i <= N) { Fr[i & 255] = bv; Poff[i] = ba >= 0 ? (uint8_t)(i - ba) : 0; }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 8; ++k) cur[k] = nxt[k];
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
  if (dm.dtype == GRACEKV_BF16) {
    hipLaunchKernelGGL(k_curvature<uint16_t>, g1, dim3(256), 0, st, dm, (const uint16_t*)hidden, ws);
    const dim3 g3((unsigned)((dm.T + GB_I - 1) / GB_I), dm.n_seg);
    hipLaunchKernelGGL(k_gram_bf16, g3, dim3(256), 0, st, dm, (const uint16_t*)hidden, ws);
  } else {
    hipLaunchKernelGGL(k_curvature<float>, g1, dim3(256), 0, st, dm, (const float*)hidden, ws);
    const dim3 g3((unsigned)((dm.T + 15) / 16), dm.n_seg);
    hipLaunchKernelGGL(k_gram_f32, g3, dim3(192), 0, st, dm, (const float*)hidden, ws);
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
