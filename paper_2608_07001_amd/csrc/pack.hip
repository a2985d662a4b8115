// Ragged compressed cache (App. A.5 "Frontier updates and physical packing",
// eq:app_frontier_update).  A node is on its tree's frontier when the op that
// created it executed (Add for the root, the parent's Split otherwise) and its
// own Split did not.  Per (l, g) the output holds, in ascending position, each
// frontier node -- a singleton as its original K/V with its position and
// log-multiplicity 0, any other node as its prototype (k~, v~ rounded to the
// cache dtype, p_v, log m_eff; App. A.3) -- followed by the r recent-window
// tokens.  A root's prototype is the one the tree build stored; deeper nodes
// are recomputed from K and V.  Offsets are a CSR over (l, g).
#include "common.h"

namespace gkv {

struct PackWs {
  int32_t* ucount;   // [unit_cap] frontier nodes per unit
  int64_t* uoff;     // [unit_cap] offset of the unit inside its (l, g) range
};

size_t pack_ws_bytes(const Dims& dm) {
  const int64_t units = (int64_t)dm.L * dm.G * dm.J_cap;
  return (size_t)units * (4 + 8) + 64;
}

static PackWs pack_view(void* ws, const Dims& dm) {
  const int64_t units = (int64_t)dm.L * dm.G * dm.J_cap;
  PackWs p;
  p.uoff = (int64_t*)ws;
  p.ucount = (int32_t*)((char*)ws + units * 8);
  return p;
}

__device__ __forceinline__ bool on_frontier(const TreeView& tv, int64_t u, int64_t base, int i) {
  const int par = tv.node_parent[base + i];
  const bool created = par < 0 ? tv.add_exec[u] != 0 : tv.sp_exec[base + par] != 0;
  if (!created) return false;
  return tv.node_nch[base + i] == 0 || tv.sp_exec[base + i] == 0;
}

__global__ void k_pack_count(Dims dm, TreeView tv, PackWs pw) {
  const int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= (int64_t)dm.L * dm.G * dm.J_cap) return;
  const int lg = (int)(u / dm.J_cap), j = (int)(u % dm.J_cap);
  const int J = *tv.nslots;
  if (j >= J) { pw.ucount[u] = 0; return; }
  const int64_t base = (int64_t)lg * 2 * dm.N_c + 2 * (int64_t)tv.slots[j];
  const int nn = tv.unit_nn[u];
  int c = 0;
  for (int i = 0; i < nn; ++i) c += on_frontier(tv, u, base, i);
  pw.ucount[u] = c;
}

// per (l, g): exclusive scan over its units, then the (l, g) entry count
__global__ __launch_bounds__(256) void k_pack_scan_units(Dims dm, TreeView tv, PackWs pw, int64_t* counts) {
  const int lg = blockIdx.x;
  const int J = *tv.nslots;
  __shared__ int64_t part[256];
  __shared__ int64_t carry;
  if (threadIdx.x == 0) carry = 0;
  __syncthreads();
  for (int j0 = 0; j0 < J; j0 += 256) {
    const int j = j0 + threadIdx.x;
    const int64_t v = j < J ? pw.ucount[(int64_t)lg * dm.J_cap + j] : 0;
    part[threadIdx.x] = v;
    __syncthreads();
    for (int o = 1; o < 256; o <<= 1) {          // inclusive Hillis-Steele scan
      const int64_t x = threadIdx.x >= o ? part[threadIdx.x - o] : 0;
      __syncthreads();
      part[threadIdx.x] += x;
      __syncthreads();
    }
    if (j < J) pw.uoff[(int64_t)lg * dm.J_cap + j] = carry + part[threadIdx.x] - v;
    __syncthreads();
    if (threadIdx.x == 0) carry += part[255];
    __syncthreads();
  }
  if (threadIdx.x == 0) counts[lg] = carry + dm.r;
}

__global__ void k_pack_scan_lg(Dims dm, const int64_t* __restrict__ counts, int64_t* offsets) {
  if (threadIdx.x != 0) return;
  int64_t acc = 0;
  offsets[0] = 0;
  for (int i = 0; i < dm.L * dm.G; ++i) {
    acc += counts[i];
    offsets[i + 1] = acc;
  }
}

// one wave per unit
template <typename T, int D>
__global__ __launch_bounds__(64) void k_pack_emit(Dims dm, const T* __restrict__ K, const T* __restrict__ V,
                                                  const float* __restrict__ cosT, const float* __restrict__ sinT,
                                                  TreeView tv, PackWs pw, const int64_t* __restrict__ offsets,
                                                  T* __restrict__ Ko, T* __restrict__ Vo, int32_t* __restrict__ po,
                                                  float* __restrict__ lo) {
  constexpr int H2 = D / 2;
  constexpr int DL = (D + 63) / 64;   // dims per lane
  const int64_t u = blockIdx.x;
  const int lg = (int)(u / dm.J_cap), j = (int)(u % dm.J_cap);
  const int J = *tv.nslots;
  if (j >= J) return;
  const int lane = threadIdx.x;
  const int64_t base = (int64_t)lg * 2 * dm.N_c + 2 * (int64_t)tv.slots[j];
  const int nn = tv.unit_nn[u];
  __shared__ int fa[NODE_MAX];
  __shared__ int fid[NODE_MAX];
  __shared__ int nf;
  __shared__ float mk[D];
  if (lane == 0) nf = 0;
  __syncthreads();
  // frontier nodes; their rank by start gives the output order
  for (int i = lane; i < nn; i += 64) fa[i] = on_frontier(tv, u, base, i) ? tv.node_a[base + i] : -1;
  __syncthreads();
  for (int i = lane; i < nn; i += 64) {
    if (fa[i] < 0) continue;
    int rank = 0;
    for (int k = 0; k < nn; ++k) rank += (fa[k] >= 0 && fa[k] < fa[i]);
    fid[rank] = i;
  }
  __syncthreads();
  const int cnt = pw.ucount[u];
  const int64_t out0 = offsets[lg] + pw.uoff[u];
  const T* Kp = K + (int64_t)lg * dm.T * D;
  const T* Vp = V + (int64_t)lg * dm.T * D;
  const float* Rt = tv.tok_R + (int64_t)lg * dm.N_c;
  for (int r = 0; r < cnt; ++r) {
    const int i = fid[r];
    const int a = tv.node_a[base + i], n = tv.node_n[base + i];
    const int64_t o = out0 + r;
    if (o >= dm.B_total) { if (lane == 0) atomicOr(tv.status, STATUS_CAPACITY); break; }
    if (n == 1) {
      for (int c = lane; c < D; c += 64) {
        Ko[o * D + c] = Kp[(int64_t)a * D + c];
        Vo[o * D + c] = Vp[(int64_t)a * D + c];
      }
      if (lane == 0) { po[o] = a; lo[o] = 0.f; }
      continue;
    }
    if (i == 0) {                             // the root: the prototype the build stored
      const T* pr = (const T*)tv.proto + u * 2 * D;
      for (int c = lane; c < D; c += 64) {
        Ko[o * D + c] = pr[c];
        Vo[o * D + c] = pr[D + c];
      }
      if (lane == 0) { po[o] = round_half_even_mid(a, a + n); lo[o] = tv.proto_logm[u]; }
      continue;
    }
    float sk[DL], srv[DL], sv[DL];
#pragma unroll
    for (int k = 0; k < DL; ++k) { sk[k] = 0.f; srv[k] = 0.f; sv[k] = 0.f; }
    float sr = 0.f, skn = 0.f;
    for (int t = a; t < a + n; ++t) {
      const float rt = Rt[t];
      float kk = 0.f;
#pragma unroll
      for (int k = 0; k < DL; ++k) {
        const int i2 = lane + 64 * k;
        if (i2 < D) {
          const int ih = i2 < H2 ? i2 : i2 - H2;
          const int ip = i2 < H2 ? i2 + H2 : i2 - H2;
          const float c = cosT[(int64_t)t * H2 + ih], s = sinT[(int64_t)t * H2 + ih];
          const float x = ldf(Kp, (int64_t)t * D + i2), y = ldf(Kp, (int64_t)t * D + ip);
          const float kr = i2 < H2 ? x * c + y * s : x * c - y * s;
          const float v = ldf(Vp, (int64_t)t * D + i2);
          sk[k] += kr;
          srv[k] += rt * v;
          sv[k] += v;
          kk += x * x;
        }
      }
      kk = wave_sum(kk);
      skn += sqrtf(kk);
      sr += rt;
    }
    const float inv = 1.0f / (float)n;
    float ss = 0.f;
#pragma unroll
    for (int k = 0; k < DL; ++k) {
      const int i2 = lane + 64 * k;
      if (i2 < D) { mk[i2] = sk[k] * inv; ss += mk[i2] * mk[i2]; }
    }
    ss = wave_sum(ss);
    __syncthreads();
    const float coh = sqrtf(ss) / (skn * inv + dm.eps);
    const float me = fminf(fmaxf((float)n * coh * coh, 1.0f), (float)n);
    int s2 = 2 * a + n - 1;
    int p = (s2 & 1) == 0 ? (s2 >> 1) : (((s2 >> 1) & 1) ? (s2 >> 1) + 1 : (s2 >> 1));
    const float beta = dm.beta_frac * sr * inv;
    const float den = sr + (float)n * beta + dm.eps;
#pragma unroll
    for (int k = 0; k < DL; ++k) {
      const int i2 = lane + 64 * k;
      if (i2 < D) {
        const int ih = i2 < H2 ? i2 : i2 - H2;
        const float c = cosT[(int64_t)p * H2 + ih], s = sinT[(int64_t)p * H2 + ih];
        const float kt = i2 < H2 ? mk[i2] * c - mk[i2 + H2] * s : mk[i2] * c + mk[i2 - H2] * s;
        stf(Ko, o * D + i2, kt);
        stf(Vo, o * D + i2, (srv[k] + beta * sv[k]) / den);
      }
    }
    if (lane == 0) { po[o] = p; lo[o] = logf(me); }
    __syncthreads();
  }
}

// recent window: tokens [N_c, N_ctx) after the frontier entries of each (l, g)
template <typename T>
__global__ void k_pack_window(Dims dm, const T* __restrict__ K, const T* __restrict__ V,
                              const int64_t* __restrict__ offsets, T* Ko, T* Vo, int32_t* po, float* lo) {
  const int lg = blockIdx.y;
  const int k = blockIdx.x;
  const int64_t t = dm.N_c + k;
  const int64_t o = offsets[lg + 1] - dm.r + k;
  if (o < 0 || o >= dm.B_total) return;
  for (int c = threadIdx.x; c < dm.d; c += blockDim.x) {
    Ko[o * dm.d + c] = K[((int64_t)lg * dm.T + t) * dm.d + c];
    Vo[o * dm.d + c] = V[((int64_t)lg * dm.T + t) * dm.d + c];
  }
  if (threadIdx.x == 0) { po[o] = (int32_t)t; lo[o] = 0.f; }
}

hipError_t launch_pack(const Dims& dm, const void* K, const void* V, const float* cosT, const float* sinT,
                       const TreeView& tv, int64_t* offsets, int64_t* counts, void* K_out, void* V_out,
                       int32_t* pos_out, float* logm_out, void* ws, hipStream_t st) {
  PackWs pw = pack_view(ws, dm);
  const int64_t units = (int64_t)dm.L * dm.G * dm.J_cap;
  const int LG = dm.L * dm.G;
  hipLaunchKernelGGL(k_pack_count, dim3((unsigned)((units + 127) / 128)), dim3(128), 0, st, dm, tv, pw);
  hipLaunchKernelGGL(k_pack_scan_units, dim3(LG), dim3(256), 0, st, dm, tv, pw, counts);
  hipLaunchKernelGGL(k_pack_scan_lg, dim3(1), dim3(64), 0, st, dm, (const int64_t*)counts, offsets);
  const int clk = clock_begin(dm, GRACEKV_STAGE_PACK, st);
#define GKV_EMIT(TT, DD)                                                                                     \
  hipLaunchKernelGGL((k_pack_emit<TT, DD>), dim3((unsigned)units), dim3(64), 0, st, dm, (const TT*)K,       \
                     (const TT*)V, cosT, sinT, tv, pw, (const int64_t*)offsets, (TT*)K_out, (TT*)V_out, pos_out, \
                     logm_out)
  if (dm.dtype == GRACEKV_BF16) {
    if (dm.d == 128) GKV_EMIT(uint16_t, 128); else GKV_EMIT(uint16_t, 64);
  } else {
    if (dm.d == 128) GKV_EMIT(float, 128); else GKV_EMIT(float, 64);
  }
#undef GKV_EMIT
  clock_end(clk, st);
  if (dm.r > 0) {
    if (dm.dtype == GRACEKV_BF16)
      hipLaunchKernelGGL(k_pack_window<uint16_t>, dim3(dm.r, LG), dim3(64), 0, st, dm, (const uint16_t*)K,
                         (const uint16_t*)V, (const int64_t*)offsets, (uint16_t*)K_out, (uint16_t*)V_out, pos_out,
                         logm_out);
    else
      hipLaunchKernelGGL(k_pack_window<float>, dim3(dm.r, LG), dim3(64), 0, st, dm, (const float*)K,
                         (const float*)V, (const int64_t*)offsets, (float*)K_out, (float*)V_out, pos_out, logm_out);
  }
  return hipGetLastError();
}

}  // namespace gkv
