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
#include <climits>

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
  double* bsum;     // [N_c / PS_BLK + 1] prefix block totals, then offsets
  double* boff;
  void* rz;         // robust-z select state
  uint8_t* Poff;    // [N_c + 1] backpointer offsets i - P(i) (0: none)
  double* Fdbg;     // [4] F(N), chunks recomputed by the fix-up
  double* S;        // [N_c][128] slot scores by (i, length), candidate-major per lane
  long long* Fg;    // [C][DPC + 128] fixed-point F of positions c DPC - 127 .. (c + 1) DPC
  long long* dlt;   // [C] offset that turns Fg[c] into the true F
  long long* cdiff; // [C] constant difference Fg[c-1] - Fg[c] over chunk c's window
  int32_t* cok;     // [C] that difference is constant
  double* smax_part; // [N_c / SLE + 1] largest finite |S| per slot-score workgroup
  int2* bt_tab;     // [C][128] backtrack: (exit, starts emitted) per chunk entry
  int2* bt_ent;     // [C] (entry, output offset) of each chunk on the path
};

// Chunk-parallel DP: ends per chunk and the warm-up margin of a chunk's guessed run.
constexpr int DPC = 1024;
constexpr int DPM = 1024;
__host__ __device__ inline int64_t dp_chunks(int64_t N) { return (N + DPC - 1) / DPC; }

static size_t al(size_t x) { return (x + 255) & ~(size_t)255; }

size_t segment_ws_bytes(const Dims& dm) {
  const size_t T = (size_t)dm.T, N = (size_t)dm.N_c, C = (size_t)dp_chunks(dm.N_c) + 1;
  return al(dm.n_seg * 3 * T * 4) + al(dm.n_seg * T * 4) + al(T * 4) + al((size_t)dm.n_seg * T * BAND * 4) +
         al(N * BAND * 4) + 2 * al((N / 2048 + 2) * 8) + al(4096) + al((N + 1) * 8) + al(N + 1) + al(4 * 8) + al(N * BAND * 8) + al(C * (DPC + 128) * 8) +
         3 * al(C * 8) + al((N / 16 + 2) * 8) + al(C * 128 * 8) + al(C * 8);
}

static SegWs seg_view(void* ws, const Dims& dm) {
  const size_t T = (size_t)dm.T, N = (size_t)dm.N_c, C = (size_t)dp_chunks(dm.N_c) + 1;
  char* p = (char*)ws;
  SegWs s;
  s.kap9 = (float*)p; p += al(dm.n_seg * 3 * T * 4);
  s.sqd = (float*)p; p += al(dm.n_seg * T * 4);
  s.sq = (float*)p; p += al(T * 4);
  s.gram = (float*)p; p += al((size_t)dm.n_seg * T * BAND * 4);
  s.dist2 = (float*)p; p += al(N * BAND * 4);
  s.bsum = (double*)p; p += al((N / 2048 + 2) * 8);
  s.boff = (double*)p; p += al((N / 2048 + 2) * 8);
  s.rz = (void*)p; p += al(4096);
  s.P2 = (double*)p; p += al((N + 1) * 8);
  s.Poff = (uint8_t*)p; p += al(N + 1);
  s.Fdbg = (double*)p; p += al(4 * 8);
  s.S = (double*)p; p += al(N * BAND * 8);
  s.Fg = (long long*)p; p += al(C * (DPC + 128) * 8);
  s.dlt = (long long*)p; p += al(C * 8);
  s.cdiff = (long long*)p; p += al(C * 8);
  s.cok = (int32_t*)p; p += al(C * 8);
  s.smax_part = (double*)p; p += al((N / 16 + 2) * 8);
  s.bt_tab = (int2*)p; p += al(C * 128 * 8);
  s.bt_ent = (int2*)p;
  return s;
}

// Thread (p, q) owns the four positions i0 + 4p .. i0 + 4p + 3 and column quad
// q of each 64-column chunk (p = lane % 16, q = 4 wave + lane / 16).  The window
// sums of the first position are built tap by tap, then slid one position at a
// time (one row in, one out per window); the partial dot products are summed
// over the four quads of a wave by row-swap permutations and over the waves in
// LDS.  Rows are scaled by 1 / max(||h||, eps) while staged, the norm taken
// from the diagonal of the banded Gram (computed first).
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
  const int pg = lane & 15, cq = wave * 4 + (lane >> 4);
  const int r0 = 4 * pg + CHALO;                    // staged row of the first position
  float acc[4][10];                                  // per position: 3 windows x (dot, |d-|^2, |d+|^2), then |h_{i+1} - h_i|^2
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int v = 0; v < 10; ++v) acc[k][v] = 0.f;
  constexpr int EPL = 16 / (int)sizeof(T);          // elements per 16-byte load
  constexpr int LPR = CCOL / EPL;                   // loads per staged row
  static_assert(CCOL / 4 == 16, "sixteen column quads per chunk");
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
    const float* col = hb + 4 * cq;
    auto ld = [&](int r) { return *(const float4*)(col + r * CLD); };
    // window sums of the first position: left [r - w + 1, r], right [r + 1, r + w]
    float4 sm[3], sp[3];
    {
      float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a;
      int tau = 0;
#pragma unroll
      for (int w = 0; w < 3; ++w) {
        const int ww = w == 0 ? 4 : (w == 1 ? 8 : 16);
#pragma unroll
        for (; tau < ww; ++tau) {
          const float4 x1 = ld(r0 - tau), x2 = ld(r0 + 1 + tau);
          a.x += x1.x; a.y += x1.y; a.z += x1.z; a.w += x1.w;
          b.x += x2.x; b.y += x2.y; b.z += x2.z; b.w += x2.w;
        }
        sm[w] = a;
        sp[w] = b;
      }
    }
    float4 xc = ld(r0);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int r = r0 + k;
      if (k > 0) {                                   // slide every window by one position
        const float4 xn = ld(r);
#pragma unroll
        for (int w = 0; w < 3; ++w) {
          const int ww = w == 0 ? 4 : (w == 1 ? 8 : 16);
          const float4 o = ld(r - ww), in = ld(r + ww);
          sm[w].x += xn.x - o.x; sm[w].y += xn.y - o.y; sm[w].z += xn.z - o.z; sm[w].w += xn.w - o.w;
          sp[w].x += in.x - xn.x; sp[w].y += in.y - xn.y; sp[w].z += in.z - xn.z; sp[w].w += in.w - xn.w;
        }
        xc = xn;
      }
      const float xv[4] = {xc.x, xc.y, xc.z, xc.w};
#pragma unroll
      for (int w = 0; w < 3; ++w) {
        const float iw = w == 0 ? 0.25f : (w == 1 ? 0.125f : 0.0625f);
        const float smv[4] = {sm[w].x, sm[w].y, sm[w].z, sm[w].w}, spv[4] = {sp[w].x, sp[w].y, sp[w].z, sp[w].w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float dmn = xv[q] - smv[q] * iw;
          const float dpl = spv[q] * iw - xv[q];
          acc[k][3 * w] += dmn * dpl;
          acc[k][3 * w + 1] += dmn * dmn;
          acc[k][3 * w + 2] += dpl * dpl;
        }
      }
      const float4 n4 = ld(r + 1);
      const float nv[4] = {n4.x, n4.y, n4.z, n4.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) { const float dd = nv[q] - xv[q]; acc[k][9] += dd * dd; }
    }
  }
  // the four quads of the wave (lanes p + 16 j), then the waves in LDS
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int v = 0; v < 10; ++v) {
      const float t = col_sum4(acc[k][v]);
      if (lane < 16) red[wave][v][4 * pg + k] = t;
    }
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

// Lower medians by a multi-workgroup radix select on order-preserving keys:
// selects 0 and 1 run together (kappa and s, then |kappa - med| and |s - med|);
// per pass every workgroup adds its 256-bin histogram of the keys matching the
// prefix, and the last one to finish picks the digit.
struct RzState {
  uint32_t prefix[2];
  int64_t rank[2];
  float center[2];
  float med[4];                 // med kappa, med s, MAD kappa, MAD s
  uint32_t done[2];
  uint32_t hist[2][256];
};
constexpr int RZ_WG = 128;      // workgroups per select and pass

__global__ void k_rz_init(Dims dm, RzState* R, int stage) {
  const int t = threadIdx.x;
  R->hist[0][t] = 0;
  R->hist[1][t] = 0;
  if (t < 2) {
    R->prefix[t] = 0;
    R->rank[t] = (dm.T - 1) / 2;
    R->done[t] = 0;
    R->center[t] = stage == 0 ? 0.f : R->med[t];
  }
}

__global__ __launch_bounds__(256) void k_rz_hist(Dims dm, const float* __restrict__ kappa,
                                                 const float* __restrict__ surp, RzState* R, int stage, int pass) {
  __shared__ uint32_t h[256];
  __shared__ bool last;
  const int which = blockIdx.y;
  const float* src = which == 0 ? kappa : surp;
  const bool absdev = stage == 1;
  const float center = R->center[which];
  const uint32_t prefix = R->prefix[which];
  const int shift = 24 - 8 * pass;
  h[threadIdx.x] = 0;
  __syncthreads();
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < dm.T; i += (int64_t)gridDim.x * 256) {
    const float v = absdev ? fabsf(src[i] - center) : src[i];
    const uint32_t k = okey(v);
    if (pass > 0 && (k >> (shift + 8)) != (prefix >> (shift + 8))) continue;
    atomicAdd(&h[(k >> shift) & 255u], 1u);
  }
  __syncthreads();
  if (h[threadIdx.x]) atomicAdd(&R->hist[which][threadIdx.x], h[threadIdx.x]);
  wait_vm();                                  // this thread's histogram atomics are performed
  __syncthreads();
  if (threadIdx.x == 0) last = atomicAdd(&R->done[which], 1u) == gridDim.x - 1;
  __syncthreads();
  if (!last) return;
  // the last workgroup: the histogram in one coalesced device-coherent read,
  // cleared for the next pass, then scanned by one thread
  h[threadIdx.x] = ld_agent(&R->hist[which][threadIdx.x]);
  R->hist[which][threadIdx.x] = 0;
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t cum = 0, rank = R->rank[which];
    for (int k = 0; k < 256; ++k) {
      const int64_t hk = h[k];
      if (cum + hk > rank) {
        R->prefix[which] = prefix | ((uint32_t)k << shift);
        R->rank[which] = rank - cum;
        break;
      }
      cum += hk;
    }
    R->done[which] = 0;
    if (pass == 3) R->med[2 * stage + which] = okey_inv(R->prefix[which]);
  }
}

__global__ void k_rz_score(Dims dm, const float* __restrict__ kappa, const float* __restrict__ surp,
                           const RzState* __restrict__ R, float* bscore) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= dm.T) return;
  const float mk = R->med[0], ms = R->med[1];
  const float dk = dm.mad * R->med[2] + dm.eps_seg, ds = dm.mad * R->med[3] + dm.eps_seg;
  bscore[i] = (kappa[i] - mk) / dk + dm.lam_s * ((surp[i] - ms) / ds);
}

// ---- K3: banded Gram --------------------------------------------------------
// bf16: a workgroup owns 64 rows i0 .. i0+63 of one slab and the 192 rows
// j in [i0 - 128, i0 + 64) they pair with; 64-dim chunks of those rows are
// staged in LDS (double-buffered, 16-byte loads) and wave w accumulates the
// 16 x 16 tiles (i-tile w, j-tile w .. w + 8) that touch the band.  A lane
// supplies 16 consecutive dims of a chunk per operand (4 k-steps), so each
// operand is two 16-byte LDS reads.
constexpr int GB_I = 128;                // rows i per workgroup (one 16-row tile per wave)
constexpr int GB_T = 4 * GB_I;           // threads per workgroup
constexpr int GB_J = GB_I + BAND;        // rows j staged
constexpr int GB_C = 64;                 // dims per chunk
constexpr int GB_LD = GB_C + 8;          // LDS row stride (bf16)

__global__ __launch_bounds__(GB_T) void k_gram_bf16(Dims dm, const uint16_t* __restrict__ hidden, SegWs ws) {
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
    for (int k = 0; k < (GB_J * CPR) / GB_T; ++k) {
      const int e = tid + GB_T * k;
      const int r = e / CPR, c = (e % CPR) * 8;
      const int64_t row = j0 + r;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (row >= 0 && row < T_ && c0 + c < Dh) v = *(const uint4*)(H + row * Dh + c0 + c);
      reg[k] = v;
    }
  };
  auto store = [&](int buf, const uint4* reg) {
#pragma unroll
    for (int k = 0; k < (GB_J * CPR) / GB_T; ++k) {
      const int e = tid + GB_T * k;
      const int r = e / CPR, c = (e % CPR) * 8;
      *(uint4*)(sh[buf] + r * GB_LD + c) = reg[k];
    }
  };
  static_assert((GB_J * CPR) % GB_T == 0, "whole staging rounds");
  uint4 reg[(GB_J * CPR) / GB_T];
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

// dist2[e][delta] = mean over slabs of ||hbar_e - hbar_{e-delta}||^2, e < N_c, from the
// banded Gram of the raw rows and their norms
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

// P2[t] = sum_{tau < t} sq[tau] (fp64), t = 0..N_c (d_t exists for t <= N_c - 2):
// block totals of PS_BLK terms, an exclusive scan of the totals, then each
// block's own scan plus its offset.
constexpr int PS_BLK = 2048;    // terms per workgroup (8 per thread)
__device__ __forceinline__ double sq_term(const Dims& dm, const SegWs& ws, int64_t t) {
  return t < dm.N_c - 1 ? (double)ws.sq[t] : 0.0;
}
__global__ __launch_bounds__(256) void k_psum_blocks(Dims dm, SegWs ws) {
  __shared__ double red[4];
  const int64_t t0 = (int64_t)blockIdx.x * PS_BLK + 8 * threadIdx.x;
  double s8 = 0.0;
#pragma unroll
  for (int k = 0; k < 8; ++k) s8 += sq_term(dm, ws, t0 + k);
  s8 = wave_sum(s8);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s8;
  __syncthreads();
  if (threadIdx.x == 0) ws.bsum[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}
__global__ __launch_bounds__(1024) void k_psum_top(Dims dm, SegWs ws, int nblk) {
  __shared__ double part[1024];
  __shared__ double carry;
  if (threadIdx.x == 0) carry = 0.0;
  __syncthreads();
  for (int b0 = 0; b0 < nblk; b0 += 1024) {
    const int b = b0 + threadIdx.x;
    const double v = b < nblk ? ws.bsum[b] : 0.0;
    part[threadIdx.x] = v;
    __syncthreads();
    for (int o = 1; o < 1024; o <<= 1) {
      const double x = threadIdx.x >= o ? part[threadIdx.x - o] : 0.0;
      __syncthreads();
      part[threadIdx.x] += x;
      __syncthreads();
    }
    if (b < nblk) ws.boff[b] = carry + part[threadIdx.x] - v;
    __syncthreads();
    if (threadIdx.x == 0) carry += part[1023];
    __syncthreads();
  }
}
__global__ __launch_bounds__(256) void k_psum_apply(Dims dm, SegWs ws) {
  __shared__ double part[256];
  const int64_t t0 = (int64_t)blockIdx.x * PS_BLK + 8 * threadIdx.x;
  double v[8], s8 = 0.0;
#pragma unroll
  for (int k = 0; k < 8; ++k) { v[k] = sq_term(dm, ws, t0 + k); s8 += v[k]; }
  part[threadIdx.x] = s8;
  __syncthreads();
  for (int o = 1; o < 256; o <<= 1) {
    const double x = threadIdx.x >= o ? part[threadIdx.x - o] : 0.0;
    __syncthreads();
    part[threadIdx.x] += x;
    __syncthreads();
  }
  double run = ws.boff[blockIdx.x] + part[threadIdx.x] - s8;   // sum of the terms before t0
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    run += v[k];
    if (t0 + k < dm.N_c) ws.P2[t0 + k + 1] = run;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) ws.P2[0] = 0.0;
}

// ---- K4: DP -----------------------------------------------------------------
// The slot score Gamma(a) - lam_d Disp([a, i)) - lam_n ((i - a - n0) / n0)^2 of
// eq:app_dp_recurrence does not depend on F: it is tabulated for every end i
// and length in parallel (fp64), then the recurrence only adds F[a] and takes
// the maximum.  Candidate c = len - n_min of end i is stored at
// S[(i - 1) * 128 + (c % 16) * 8 + c / 16], so the lane that owns candidates
// c = sub, sub + 16, ... reads 8 consecutive doubles.
//
// The recurrence runs in fixed point: every score is rounded once to an
// integer multiple of 2^-e (e chosen from the largest |S| so that no F can
// overflow 2^60), after which additions are exact and associative.  That makes
// the chunk-parallel form below give bit for bit the result of the serial
// recurrence on the same integers, ties included:
//   * the ends are cut into chunks of DPC; every chunk runs the recurrence from
//     a guessed state DPM positions before it (all F there = 0), all chunks at
//     once;
//   * if the guessed F over the 128 positions a chunk's ends can reach back to
//     differ from the true F there by one constant, every F of the chunk
//     differs by that constant and every backpointer is the true one (adding a
//     constant to all predecessors changes neither the maximum's position nor
//     its ties);
//   * a check kernel tests that condition for all chunks in parallel against
//     the previous chunk's guess, and a one-workgroup pass chains the
//     constants and recomputes, from the true state, any chunk that fails.
// Ties go to the smallest predecessor; terminal relaxation
// eq:app_terminal_predecessor; backtrack from LDS.
constexpr long long DP_NEG = LLONG_MIN / 2;    // unreachable

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

// SLE ends per workgroup, one candidate length per thread; the workgroup's
// largest finite |S| goes to smax_part (reduced by the DP kernels).
constexpr int SLE = 16;
__global__ __launch_bounds__(128) void k_slot_scores(Dims dm, const float* __restrict__ b, SegWs ws) {
  __shared__ double red[2];
  const int c = threadIdx.x;
  const int len = dm.n_min + c;
  double m = 0.0;
  for (int k = 0; k < SLE; ++k) {
    const int64_t i = (int64_t)blockIdx.x * SLE + k + 1;
    if (i > dm.N_c) break;
    double v = -INFINITY;
    if (len <= dm.n_max && i - len >= 0) v = slot_score(dm, b, ws, i, len);
    ws.S[(i - 1) * BAND + (c % 16) * 8 + c / 16] = v;
    if (isfinite(v)) m = fmax(m, fabs(v));
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) m = fmax(m, __shfl_xor(m, o, 64));
  if ((c & 63) == 0) red[c >> 6] = m;
  __syncthreads();
  if (c == 0) ws.smax_part[blockIdx.x] = fmax(red[0], red[1]);
}

// largest finite |S| over the slot-score workgroups (every thread gets it)
__device__ double dp_smax(const Dims& dm, const SegWs& ws) {
  __shared__ double red[16];
  const int64_t nb = (dm.N_c + SLE - 1) / SLE;
  double m = 0.0;
  for (int64_t k = threadIdx.x; k < nb; k += blockDim.x) m = fmax(m, ws.smax_part[k]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) m = fmax(m, __shfl_xor(m, o, 64));
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  double r = 0.0;
  for (int w = 0; w < (int)(blockDim.x + 63) / 64; ++w) r = fmax(r, red[w]);
  __syncthreads();
  return r;
}

// 2^e with (max |S| + 1) (N / n_min + 2) 2^e < 2^60 (every thread of the workgroup calls it)
__device__ __forceinline__ double dp_scale(const Dims& dm, const SegWs& ws) {
  const double mx = dp_smax(dm, ws);
  const double bound = (mx + 1.0) * (double)(dm.N_c / dm.n_min + 2);
  int e = 0;
  frexp(bound, &e);                            // bound < 2^e
  int sh = 60 - e;
  if (sh > 48) sh = 48;
  return ldexp(1.0, sh);
}
__device__ __forceinline__ long long dp_fix(double s, double sc) {
  return isfinite(s) ? (long long)__double2ll_rn(s * sc) : DP_NEG;
}

// one DPP step of the (value, smallest start) maximum within 16-lane rows
// (an absent candidate is (DP_NEG, INT_MAX) and never wins)
template <int CTRL>
__device__ __forceinline__ void dp_step(long long& bv, int& ba) {
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(bv & 0xffffffffll), CTRL, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(bv >> 32), CTRL, 0xf, 0xf, false);
  const int a2 = __builtin_amdgcn_update_dpp(0, ba, CTRL, 0xf, 0xf, false);
  const long long v2 = ((long long)hi << 32) | (long long)(unsigned)lo;
  const bool better = v2 > bv || (v2 == bv && a2 < ba);
  bv = better ? v2 : bv;
  ba = better ? a2 : ba;
}
// every lane of a 16-lane row ends with the row's best: lanes ^1, ^2 (quad
// permutes), then rotations by 4 and 8 within the row
__device__ __forceinline__ void dp_reduce16(long long& bv, int& ba) {
  dp_step<0xB1>(bv, ba);     // quad_perm(1, 0, 3, 2)
  dp_step<0x4E>(bv, ba);     // quad_perm(2, 3, 0, 1)
  dp_step<0x124>(bv, ba);    // row_ror:4
  dp_step<0x128>(bv, ba);    // row_ror:8
}

// F of the ends lo .. hi (inclusive), 256 threads: with n_min >= 16,
// F[i .. i+15] depend only on F[< i], so wave w owns ends i0 + 4 w .. i0 + 4 w + 3
// of a step, 16 lanes per end, each lane 8 candidate lengths.  Fr (LDS ring,
// index position & 255) holds F of positions lo - 128 .. lo - 1 on entry.
// Backpointer offsets go to Poff for ends >= own_lo; F of positions >= fg_lo
// to Fg[position - fg_lo].
__device__ void dp_run(const Dims& dm, const SegWs& ws, double sc, long long* Fr, int64_t lo, int64_t hi,
                       int64_t own_lo, long long* Fg, int64_t fg_lo) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int st = lane >> 4, sub = lane & 15;
  // unconditional loads (row clamped to hi) keep the load counter exact
  auto load = [&](int64_t i, double* sv) {
    const int64_t ic = i <= hi ? i : hi;
    const double2* p = (const double2*)(ws.S + (ic - 1) * BAND + sub * 8);
#pragma unroll
    for (int k = 0; k < 4; ++k) { const double2 v = p[k]; sv[2 * k] = v.x; sv[2 * k + 1] = v.y; }
  };
  // scores of 4 steps in flight (static register indices: the step loop is unrolled by 4)
  double sv[4][8];
#pragma unroll
  for (int q = 0; q < 4; ++q) load(lo + 16 * q + 4 * wave + st, sv[q]);
  for (int64_t i00 = lo; i00 <= hi; i00 += 64) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t i0 = i00 + 16 * q;
      if (i0 > hi) break;
      const int64_t i = i0 + 4 * wave + st;
      // all F reads first, then a branch-free (value, smallest start) maximum
      long long Fa[8];
      int av[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int len = dm.n_min + sub + 16 * k;
        const int64_t a = i - len;
        const bool ok = i <= hi && len <= dm.n_max && a >= 0;
        av[k] = ok ? (int)a : 0x7fffffff;
        Fa[k] = Fr[ok ? (int)(a & 255) : 0];
      }
      long long bv = DP_NEG;
      int ba = 0x7fffffff;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const long long s = dp_fix(sv[q][k], sc);
        const bool ok = av[k] != 0x7fffffff && Fa[k] != DP_NEG && s != DP_NEG;
        const long long v = ok ? Fa[k] + s : DP_NEG;
        const int a = ok ? av[k] : 0x7fffffff;
        const bool better = v > bv || (v == bv && a < ba);
        bv = better ? v : bv;
        ba = better ? a : ba;
      }
      load(i + 64, sv[q]);                   // the same lane's end four steps later
      dp_reduce16(bv, ba);
      lds_barrier();                         // every end of this step has read its F
      if (sub == 0 && i <= hi) {
        Fr[i & 255] = bv;
        if (i >= own_lo) ws.Poff[i] = ba != 0x7fffffff ? (uint8_t)(i - ba) : 0;
        if (Fg != nullptr && i >= fg_lo) Fg[i - fg_lo] = bv;
      }
      lds_barrier();
    }
  }
}

// Guessed run of chunk c = blockIdx.x: ends c DPC + 1 .. min((c + 1) DPC, N),
// warmed up from F = 0 at the 128 positions before max(c DPC - DPM, 0) (from
// the true start F[0] = 0 when that is position 0).
__global__ __launch_bounds__(256) void k_dp_chunk(Dims dm, SegWs ws) {
  __shared__ long long Fr[256];
  const int64_t N = dm.N_c;
  const int64_t c = blockIdx.x;
  const int64_t lo = c * DPC + 1, hi = (c + 1) * DPC < N ? (c + 1) * DPC : N;
  const int64_t margin = dm.dp_serial ? 0 : DPM;
  const int64_t s = c * DPC - margin > 0 ? c * DPC - margin : 0;
  const double sc = dp_scale(dm, ws);
  long long* Fg = ws.Fg + c * (DPC + 128);
  const int64_t fg_lo = c * DPC - 127;
  // ring: positions s - 127 .. s (guess 0, or the true start)
  Fr[threadIdx.x] = s == 0 ? DP_NEG : 0;
  __syncthreads();
  if (threadIdx.x == 0) {
    if (s == 0) Fr[0] = 0;
    if (c == 0) ws.Poff[0] = 0;
  }
  if (threadIdx.x < 128) {                   // window positions the run does not reach
    const int64_t pos = fg_lo + threadIdx.x;
    if (pos <= s) Fg[threadIdx.x] = pos < 0 ? DP_NEG : (s == 0 ? (pos == 0 ? 0 : DP_NEG) : 0);
  }
  __syncthreads();
  dp_run(dm, ws, sc, Fr, s + 1, hi, lo, Fg, fg_lo);
}

// For chunks c >= 1: is Fg[c-1] - Fg[c] one constant over positions
// c DPC - 127 .. c DPC (all ends of chunk c-1, since DPC >= 128)?
__global__ __launch_bounds__(128) void k_dp_check(Dims dm, SegWs ws) {
  __shared__ long long mn[2], mx[2];
  __shared__ int bad[2];
  const int64_t c = (int64_t)blockIdx.x + 1;
  const int t = threadIdx.x, w = t >> 6;
  const long long a = ws.Fg[(c - 1) * (DPC + 128) + DPC + t];   // position c DPC - 127 + t
  const long long b = ws.Fg[c * (DPC + 128) + t];
  const bool ng = a == DP_NEG || b == DP_NEG;
  long long d = a - b, dn = d, dx = d;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    dn = min(dn, (long long)__shfl_xor(dn, o, 64));
    dx = max(dx, (long long)__shfl_xor(dx, o, 64));
  }
  const bool anyng = __any(ng);
  if ((t & 63) == 0) { mn[w] = dn; mx[w] = dx; bad[w] = anyng; }
  __syncthreads();
  if (t == 0) {
    const long long n0 = min(mn[0], mn[1]), x0 = max(mx[0], mx[1]);
    ws.cok[c] = (n0 == x0 && !bad[0] && !bad[1]) ? 1 : 0;
    ws.cdiff[c] = n0;
  }
}

// Chains the chunk offsets, recomputes failing chunks from the true state,
// then the terminal relaxation (one workgroup).
__global__ __launch_bounds__(256) void k_dp_fix(Dims dm, const float* __restrict__ b, SegWs ws) {
  __shared__ long long Fr[256];
  __shared__ long long red[4];
  __shared__ int flags[4];
  __shared__ long long cur;
  const int64_t N = dm.N_c;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const double sc = dp_scale(dm, ws);
  const int64_t C = dp_chunks(N);
  auto Fg = [&](int64_t c) { return ws.Fg + c * (DPC + 128); };
  long long Dprev = 0;                         // chunk 0 starts at the true F[0] = 0
  bool dirty = false;                          // chunk c-1 was recomputed: recheck c here
  int nfix = 0;
  if (tid == 0) ws.dlt[0] = 0;
  __shared__ long long tdiff[256];
  __shared__ int tok[256];
  for (int64_t c = 1; c < C; ++c) {
    if ((c - 1) % 256 == 0) {                  // stage the check results of the next 256 chunks
      __syncthreads();
      if (c + tid < C) { tok[tid] = ws.cok[c + tid]; tdiff[tid] = ws.cdiff[c + tid]; }
      __syncthreads();
    }
    const int tc = (int)((c - 1) % 256);
    if (!dirty && tok[tc]) {
      Dprev += tdiff[tc];
      if (tid == 0) ws.dlt[c] = Dprev;
      continue;
    }
    // check against the true F of chunk c-1 (Fg + Dprev)
    long long dlo = LLONG_MAX, dhi = LLONG_MIN;
    int ng = 0;
    if (tid < 128) {
      const long long a = Fg(c - 1)[DPC + tid], g = Fg(c)[tid];
      ng = a == DP_NEG || g == DP_NEG;
      const long long d = a + Dprev - g;
      dlo = d; dhi = d;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      dlo = min(dlo, (long long)__shfl_xor(dlo, o, 64));
      dhi = max(dhi, (long long)__shfl_xor(dhi, o, 64));
    }
    const bool ngw = __any(ng);
    __syncthreads();
    if (lane == 0 && wave < 2) { red[wave] = dlo; red[2 + wave] = dhi; flags[wave] = ngw; }
    __syncthreads();
    const long long lo2 = min(red[0], red[1]), hi2 = max(red[2], red[3]);
    if (lo2 == hi2 && !flags[0] && !flags[1]) {
      Dprev = lo2;
      dirty = false;
      if (tid == 0) ws.dlt[c] = Dprev;
      continue;
    }
    // recompute chunk c from the true state; its Fg then holds true values
    if (tid < 128) {
      const int64_t pos = c * DPC - 127 + tid;
      const long long a = Fg(c - 1)[DPC + tid];
      Fr[pos & 255] = a == DP_NEG ? DP_NEG : a + Dprev;
    }
    __syncthreads();
    const int64_t lo = c * DPC + 1, hi = (c + 1) * DPC < N ? (c + 1) * DPC : N;
    dp_run(dm, ws, sc, Fr, lo, hi, lo, Fg(c), c * DPC - 127);
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");   // one workgroup: its global writes, visible to itself
    __syncthreads();
    Dprev = 0;
    dirty = true;
    ++nfix;
    if (tid == 0) ws.dlt[c] = 0;
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");   // one workgroup: its global writes, visible to itself
  __syncthreads();
  // true F at position p (p >= 0)
  auto Ftrue = [&](int64_t p) -> long long {
    if (p == 0) return 0;
    const int64_t c = (p - 1) / DPC;
    const long long v = Fg(c)[p - (c * DPC - 127)];
    return v == DP_NEG ? DP_NEG : v + ws.dlt[c];
  };
  // terminal relaxation of the last slot's minimum length
  if (ws.Poff[N] == 0 && wave == 0) {
    long long bv = DP_NEG;
    int ba = 0x7fffffff;
    for (int len = 1 + lane; len <= dm.n_max; len += 64) {
      const int64_t a = N - len;
      if (a < 0) continue;
      const long long Fa = Ftrue(a);
      if (Fa == DP_NEG) continue;
      const long long s = dp_fix(slot_score(dm, b, ws, N, len), sc);
      if (s == DP_NEG) continue;
      const long long v = Fa + s;
      if (v > bv || (v == bv && (int)a < ba)) { bv = v; ba = (int)a; }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const long long v2 = __shfl_xor(bv, o, 64);
      const int a2 = __shfl_xor(ba, o, 64);
      if (v2 > bv || (v2 == bv && a2 < ba)) { bv = v2; ba = a2; }
    }
    if (lane == 0) {
      ws.Poff[N] = ba != 0x7fffffff ? (uint8_t)(N - ba) : 0;
      cur = bv;
    }
  } else if (tid == 0) {
    cur = Ftrue(N);
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");   // one workgroup: its global writes, visible to itself
  __syncthreads();
  if (tid == 0) {
    ws.Fdbg[0] = (double)cur / sc;
    ws.Fdbg[1] = (double)nfix;
  }
}

// Uniform slots of n0 tokens, the last one shorter (ablation without the
// curvature-guided partition): starts 0, n0, 2 n0, ..., then N_c.
__global__ void k_uniform_slots(Dims dm, int32_t* slots, int32_t* nslots) {
  const int64_t J = (dm.N_c + dm.n0 - 1) / dm.n0;
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j <= J; j += (int64_t)gridDim.x * blockDim.x)
    slots[j] = (int32_t)(j < J ? j * dm.n0 : dm.N_c);
  if (blockIdx.x == 0 && threadIdx.x == 0) *nslots = (int32_t)J;
}

__global__ void k_seg_empty(int32_t* slots, int32_t* nslots) {
  if (threadIdx.x == 0) { slots[0] = 0; *nslots = 0; }
}

// ---- backtrack, chunk-parallel ---------------------------------------------
// The path N = x_0 > x_1 > ... > x_J = 0 follows x_{m+1} = x_m - Poff[x_m]; the
// slot starts are x_1 .. x_J.  A path node of chunk c (ends c DPC + 1 ..
// (c + 1) DPC) is entered from the chunk above at one of its 128 top positions
// (a slot is at most 128 long), so: every chunk walks from each of its 128
// possible entries down to its exit (the first start <= c DPC, the entry of
// chunk c - 1), counting the starts it emits; one thread chains the entries
// from N down; every chunk then re-walks from its true entry and writes its
// starts at the offset the chain gives.
__device__ __forceinline__ int bt_stage(const SegWs& ws, int64_t c, int64_t N, uint8_t* P) {
  // P[k] = Poff[c DPC + 1 + k], k < DPC
  const int64_t lo = c * DPC + 1;
  const int n = (int)((c + 1) * DPC < N ? DPC : N - c * DPC);
  for (int k = threadIdx.x; k < n; k += blockDim.x) P[k] = ws.Poff[lo + k];
  __syncthreads();
  return n;
}

// walk of chunk c from entry position e: (exit position or -1 if the path
// breaks, starts emitted)
__device__ __forceinline__ int2 bt_walk(int64_t c, const uint8_t* P, int64_t e) {
  int64_t p = e;
  int cnt = 0;
  while (p > c * DPC) {
    const int o = P[p - c * DPC - 1];
    if (o == 0) return make_int2(-1, cnt);
    p -= o;
    ++cnt;
  }
  return make_int2((int)p, cnt);
}

// bt_tab[c * 128 + k] = (exit, count) of chunk c from entry (c + 1) DPC - 127 + k
// (the last chunk: entry N, k = 0)
__global__ __launch_bounds__(128) void k_bt_walk(Dims dm, SegWs ws) {
  __shared__ uint8_t P[DPC];
  const int64_t N = dm.N_c, C = dp_chunks(N);
  const int64_t c = blockIdx.x;
  bt_stage(ws, c, N, P);
  const int k = threadIdx.x;
  int64_t e = (c + 1) * DPC - 127 + k;
  if (c == C - 1) {
    if (k != 0) return;
    e = N;
  }
  ws.bt_tab[c * 128 + k] = e > c * DPC ? bt_walk(c, P, e) : make_int2(-1, 0);
}

// entries and output offsets of every chunk, J, slots[J] = N (one thread)
__global__ void k_bt_chain(Dims dm, SegWs ws, int32_t* slots, int32_t* nslots) {
  if (threadIdx.x != 0) return;
  const int64_t N = dm.N_c, C = dp_chunks(N);
  int64_t e = N;
  int total = 0;
  for (int64_t c = C - 1; c >= 0; --c) {
    int k = c == C - 1 ? 0 : (int)(e - ((c + 1) * DPC - 127));
    if (e <= 0 || k < 0 || k >= 128) {       // the path ended (or broke) above this chunk
      ws.bt_ent[c] = make_int2(-1, 0);
      e = -1;
      continue;
    }
    const int2 t = ws.bt_tab[c * 128 + k];
    ws.bt_ent[c] = make_int2((int)e, total);
    total += t.y;
    e = t.x;
  }
  slots[total] = (int32_t)N;
  *nslots = total;
}

// chunk c re-walks from its entry; the m-th start it emits is slots[J - 1 - (offset + m)]
__global__ __launch_bounds__(64) void k_bt_emit(Dims dm, SegWs ws, int32_t* slots, const int32_t* nslots) {
  __shared__ uint8_t P[DPC];
  const int64_t N = dm.N_c;
  const int64_t c = blockIdx.x;
  const int2 ent = ws.bt_ent[c];
  if (ent.x < 0) return;
  bt_stage(ws, c, N, P);
  if (threadIdx.x != 0) return;
  const int J = *nslots;
  int64_t p = ent.x;
  int m = ent.y;
  while (p > c * DPC) {
    const int o = P[p - c * DPC - 1];
    if (o == 0) break;
    p -= o;
    slots[J - 1 - m] = (int32_t)p;
    ++m;
  }
}

hipError_t launch_segment(const Dims& dm, const void* hidden, const float* surprisal, float* kappa, float* bscore,
                          int32_t* slot_starts, int32_t* n_slots, void* wsp, hipStream_t st) {
  SegWs ws = seg_view(wsp, dm);
  const dim3 g1((unsigned)((dm.T + CT - 1) / CT), dm.n_seg);
  // the Gram first: its diagonal gives the row norms of the curvature pass
  if (dm.dtype == GRACEKV_BF16) {
    const dim3 g3((unsigned)((dm.T + GB_I - 1) / GB_I), dm.n_seg);
    hipLaunchKernelGGL(k_gram_bf16, g3, dim3(GB_T), 0, st, dm, (const uint16_t*)hidden, ws);
    hipLaunchKernelGGL(k_curvature<uint16_t>, g1, dim3(256), 0, st, dm, (const uint16_t*)hidden, ws);
  } else {
    const dim3 g3((unsigned)((dm.T + 15) / 16), dm.n_seg);
    hipLaunchKernelGGL(k_gram_f32, g3, dim3(192), 0, st, dm, (const float*)hidden, ws);
    hipLaunchKernelGGL(k_curvature<float>, g1, dim3(256), 0, st, dm, (const float*)hidden, ws);
  }
  hipLaunchKernelGGL(k_stabilize, dim3((unsigned)((dm.T + 255) / 256)), dim3(256), 0, st, dm, ws, kappa);
  {
    RzState* R = (RzState*)ws.rz;
    for (int stage = 0; stage < 2; ++stage) {
      hipLaunchKernelGGL(k_rz_init, dim3(1), dim3(256), 0, st, dm, R, stage);
      for (int pass = 0; pass < 4; ++pass)
        hipLaunchKernelGGL(k_rz_hist, dim3(RZ_WG, 2), dim3(256), 0, st, dm, (const float*)kappa, surprisal, R, stage,
                           pass);
    }
    hipLaunchKernelGGL(k_rz_score, dim3((unsigned)((dm.T + 255) / 256)), dim3(256), 0, st, dm, (const float*)kappa,
                       surprisal, (const RzState*)R, bscore);
  }
  if (dm.N_c > 0 && dm.uniform_slots) {
    const int64_t J = (dm.N_c + dm.n0 - 1) / dm.n0;
    hipLaunchKernelGGL(k_uniform_slots, dim3((unsigned)((J + 256) / 256)), dim3(256), 0, st, dm, slot_starts, n_slots);
    return hipGetLastError();
  }
  if (dm.N_c > 0) {
    hipLaunchKernelGGL(k_dist2, dim3((unsigned)dm.N_c), dim3(BAND), 0, st, dm, ws);
    const int nblk = (int)((dm.N_c + PS_BLK - 1) / PS_BLK);
    hipLaunchKernelGGL(k_psum_blocks, dim3(nblk), dim3(256), 0, st, dm, ws);
    hipLaunchKernelGGL(k_psum_top, dim3(1), dim3(1024), 0, st, dm, ws, nblk);
    hipLaunchKernelGGL(k_psum_apply, dim3(nblk), dim3(256), 0, st, dm, ws);
  }
  if (dm.N_c > 0) {
    const int64_t C = dp_chunks(dm.N_c);
    hipLaunchKernelGGL(k_slot_scores, dim3((unsigned)((dm.N_c + SLE - 1) / SLE)), dim3(BAND), 0, st, dm,
                       (const float*)bscore, ws);
    hipLaunchKernelGGL(k_dp_chunk, dim3((unsigned)C), dim3(256), 0, st, dm, ws);
    if (C > 1) hipLaunchKernelGGL(k_dp_check, dim3((unsigned)(C - 1)), dim3(128), 0, st, dm, ws);
    hipLaunchKernelGGL(k_dp_fix, dim3(1), dim3(256), 0, st, dm, (const float*)bscore, ws);
    hipLaunchKernelGGL(k_bt_walk, dim3((unsigned)C), dim3(128), 0, st, dm, ws);
    hipLaunchKernelGGL(k_bt_chain, dim3(1), dim3(64), 0, st, dm, ws, slot_starts, n_slots);
    hipLaunchKernelGGL(k_bt_emit, dim3((unsigned)C), dim3(64), 0, st, dm, ws, slot_starts, (const int32_t*)n_slots);
  } else {
    hipLaunchKernelGGL(k_seg_empty, dim3(1), dim3(64), 0, st, slot_starts, n_slots);
  }
  return hipGetLastError();
}

}  // namespace gkv
