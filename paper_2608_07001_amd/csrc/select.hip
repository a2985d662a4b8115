// Gains, keys and the global budgeted auction.
//
// Score (App. A.5 eq:app_operation_gains, eq:app_operation_costs,
// eq:app_unit_utility; eq:app_head_sensitivity; gains clamped at zero as in
// App. C.5):  Add(l,g,j): Delta = w R(root) (D_drop(root) - D(root)), cost 1;
// Split(v): Delta = w R(v) (D(v) - sum_children D), cost |child| - 1;
// U = max(Delta, 0) / c.  Every op gets the unique key
//   k = (bits(U) << 32) | (2^32 - 1 - id),  id = unit_ordinal * 256 + local,
// (larger U first, then the smaller id) and the effective key
//   E(a) = min(k(a), E(parent op)).
//
// Select (App. A.5 Stage II and App. C.3: pop the best available op, execute
// it if it fits, discard it otherwise, expose its children).  While at least
// two budget units remain every pop executes, and the queue pops ops in
// descending E (an op can only be popped after every ancestor, and once the
// queue top drops below v every op with E > v has been popped).  Hence, with
// theta the E value at which the cumulative cost in descending-E order first
// reaches B_free - 1:
//   * every op with E > theta executes;
//   * the ops with E == theta share one minimising ancestor, so they lie in
//     one unit; the queue rule is replayed there while >= 2 units remain;
//   * if exactly one unit remains, the queue discards cost-2 ops until it pops
//     a cost-1 op, i.e. it executes the best-keyed available cost-1 op.
// theta is found with an 8-pass, 8-bit, cost-weighted radix select (the last
// seven passes over a compact list of the ops that have a cost).
#include <algorithm>

#include "common.h"

namespace gkv {

enum { SEL_SELECT = 0, SEL_ALL = 1, SEL_NONE = 2, SEL_RESID = 3 };

struct SelState {
  uint64_t prefix;
  int64_t target;
  int64_t above;
  int64_t total;
  int64_t R;
  uint64_t resid_key;
  int32_t mode;
  uint32_t done;        // workgroups finished with the current pass (the last one scans)
  uint64_t ncand;       // ops in the candidate list (> cap: the list is not used)
  int64_t B;            // the auction's budget: B_free less the singleton floor's spending
  int64_t floor;        // the floor's spending B_floor
  unsigned long long hist[256];
};

// After the first pass over the whole op table the remaining passes read a
// compact list of the ops with nonzero cost: (E, cost) pairs.
constexpr int SEL_GRID = 4096;
__host__ __device__ inline int64_t sel_ops(const Dims& dm) { return (int64_t)dm.L * dm.G * 2 * dm.N_c + (int64_t)dm.L * dm.G * dm.J_cap; }
static int64_t sel_cap(const Dims& dm) { return std::min<int64_t>(sel_ops(dm), (int64_t)1 << 23); }
static size_t al256s(size_t x) { return (x + 255) & ~(size_t)255; }
size_t selstate_bytes(const Dims& dm) {
  const size_t cap = (size_t)sel_cap(dm);
  return al256s(sizeof(SelState)) + al256s(cap * 8) + al256s(cap);
}
size_t select_ws_bytes(const Dims& dm) { return selstate_bytes(dm); }
struct SelList {
  uint64_t* E;
  uint8_t* c;
  int64_t cap;
};
static SelList sel_list(void* state, const Dims& dm) {
  const size_t cap = (size_t)sel_cap(dm);
  char* p = (char*)state + al256s(sizeof(SelState));
  SelList L;
  L.E = (uint64_t*)p; p += al256s(cap * 8);
  L.c = (uint8_t*)p;
  L.cap = (int64_t)cap;
  return L;
}

__device__ __forceinline__ uint64_t make_key(float U, uint32_t id) { return op_key(U, id); }

__global__ void k_omega(Dims dm, const float* __restrict__ omega_raw, TreeView tv) {
  __shared__ float red[256];
  const int LG = dm.L * dm.G;
  float s = 0.f;
  for (int i = threadIdx.x; i < LG; i += 256) s += omega_raw ? omega_raw[i] : 1.0f;
  red[threadIdx.x] = s;
  __syncthreads();
  for (int k = 128; k > 0; k >>= 1) {
    if (threadIdx.x < k) red[threadIdx.x] += red[threadIdx.x + k];
    __syncthreads();
  }
  const float mean = red[0] / (float)LG;
  for (int i = threadIdx.x; i < LG; i += 256) tv.omega[i] = (omega_raw ? omega_raw[i] : 1.0f) / (mean + dm.eps);
}

__global__ void k_score(Dims dm, TreeView tv) {
  const int32_t* n_slots = tv.nslots;
  const int32_t* slot_starts = tv.slots;
  const int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= (int64_t)dm.L * dm.G * dm.J_cap) return;
  const int lg = (int)(u / dm.J_cap), j = (int)(u % dm.J_cap);
  const int J = *n_slots;
  if (j >= J) return;
  const uint32_t ord = (uint32_t)lg * (uint32_t)J + (uint32_t)j;
  const float w = tv.omega[lg];
  const int64_t base = (int64_t)lg * 2 * dm.N_c + 2 * (int64_t)slot_starts[j];
  const int nn = tv.unit_nn[u];
  if (nn < 1) { tv.add_U[u] = 0.f; tv.add_E[u] = 0; tv.add_exec[u] = 0; return; }
  bool bad = false;
  const float gain = add_gain(w, tv.node_R[base], tv.unit_Ddrop[u], tv.node_D[base]);
  bad |= gain != gain;
  const float Ua = utility(gain, 1);
  const uint64_t kadd = make_key(Ua, ord * 256u);
  tv.add_U[u] = Ua;
  tv.add_E[u] = kadd;
  tv.add_exec[u] = 0;
  for (int i = 0; i < nn; ++i) {
    const int64_t s = base + i;
    const int nch = tv.node_nch[s];
    tv.sp_exec[s] = 0;
    if (nch == 0) {
      tv.sp_cost[s] = 0;
      tv.sp_E[s] = 0;
      tv.sp_U[s] = 0.f;
      continue;
    }
    const int c0 = tv.node_child[s];
    float sd = 0.f;
    for (int k = 0; k < nch; ++k) sd += tv.node_D[base + c0 + k];
    const float g = split_gain(w, tv.node_R[s], tv.node_D[s], sd);
    bad |= g != g;
    const float Uv = utility(g, nch - 1);
    const uint64_t k = make_key(Uv, ord * 256u + 1u + (uint32_t)i);
    const int par = tv.node_parent[s];
    const uint64_t Ep = par < 0 ? kadd : tv.sp_E[base + par];
    tv.sp_E[s] = k < Ep ? k : Ep;
    tv.sp_U[s] = Uv;
    tv.sp_cost[s] = (uint8_t)(nch - 1);
  }
  if (bad) atomicOr(tv.status, STATUS_NUMERIC);
}

hipError_t launch_omega(const Dims& dm, const float* omega_raw, const TreeView& tv, hipStream_t st) {
  hipLaunchKernelGGL(k_omega, dim3(1), dim3(256), 0, st, dm, omega_raw, tv);
  return hipGetLastError();
}

hipError_t launch_score(const Dims& dm, const float* omega_raw, const TreeView& tv, hipStream_t st) {
  hipLaunchKernelGGL(k_omega, dim3(1), dim3(256), 0, st, dm, omega_raw, tv);
  const int64_t units = (int64_t)dm.L * dm.G * dm.J_cap;
  hipLaunchKernelGGL(k_score, dim3((unsigned)((units + 127) / 128)), dim3(128), 0, st, dm, tv);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
__global__ void k_sel_init(Dims dm, SelState* S, int rank_extra, const int64_t* fstate) {
  const int t = threadIdx.x;
  S->hist[t] = 0;
  if (t == 0) {
    S->floor = fstate ? fstate[0] : 0;
    S->B = dm.B_free - S->floor;
    S->prefix = 0; S->target = S->B - 1 + rank_extra; S->above = 0; S->total = 0; S->R = 0;
    S->resid_key = 0; S->mode = SEL_SELECT; S->done = 0; S->ncand = 0;
  }
}

// Chooses the digit of pass `pass` from the complete histogram hist (a copy in
// LDS; one thread).
__device__ void sel_scan(const Dims& dm, SelState* S, int pass, const unsigned long long* hist) {
  do {
    if (S->mode != SEL_SELECT) break;
    if (pass == 0) {
      int64_t tot = 0;
      for (int k = 0; k < 256; ++k) tot += (int64_t)hist[k];
      S->total = tot;
      if (S->B <= 0) { S->mode = SEL_NONE; break; }
      if (tot <= S->B) { S->mode = SEL_ALL; break; }
      if (S->B == 1) { S->mode = SEL_RESID; S->R = 1; break; }
    }
    const int shift = 56 - 8 * pass;
    const int64_t need = S->target - S->above;
    int64_t cum = 0;
    for (int k = 255; k >= 0; --k) {
      const int64_t hk = (int64_t)hist[k];
      if (cum + hk >= need) {
        S->prefix |= (uint64_t)k << shift;
        S->above += cum;
        break;
      }
      cum += hk;
    }
  } while (0);
  S->done = 0;
}

// cost-weighted histogram of digit `pass` among ops matching the prefix.
// Pass 0 reads the whole op table and also collects the ops that have a cost
// into a compact list (each workgroup buffers its share in LDS and appends it
// with one atomic; a workgroup whose share overflows the buffer invalidates the
// list, and the later passes then read the whole table again).  The last
// workgroup to finish a pass chooses its digit.
constexpr int SEL_BUF = 4096;
__global__ __launch_bounds__(256) void k_sel_hist(Dims dm, TreeView tv, SelState* S, int pass, SelList Lc) {
  const int32_t* n_slots = tv.nslots;
  __shared__ unsigned int h[4][256];          // one histogram per wave (less atomic contention)
  __shared__ uint64_t bufE[SEL_BUF];
  __shared__ uint8_t bufC[SEL_BUF];
  __shared__ unsigned int nbuf;
  __shared__ unsigned long long lbase;
  __shared__ bool last;
  const int tid = threadIdx.x, wave = tid >> 6;
#pragma unroll
  for (int w = 0; w < 4; ++w) h[w][tid] = 0;
  if (tid == 0) nbuf = 0;
  __syncthreads();
  const int mode = S->mode;
  const int shift = 56 - 8 * pass;
  const uint64_t pre = S->prefix;
  const int64_t ncand = (int64_t)S->ncand;
  auto take = [&](uint64_t E, int c) {
    if (pass == 0) {
      const unsigned pos = atomicAdd(&nbuf, 1u);
      if (pos < SEL_BUF) { bufE[pos] = E; bufC[pos] = (uint8_t)c; }
    }
    if (pass > 0 && (E >> (shift + 8)) != (pre >> (shift + 8))) return;
    atomicAdd(&h[wave][(E >> shift) & 255u], (unsigned)c);
  };
  if (mode == SEL_SELECT && pass > 0 && ncand <= Lc.cap) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + tid; i < ncand; i += (int64_t)gridDim.x * 256) {
      const uint64_t E = Lc.E[i];
      if ((E >> (shift + 8)) != (pre >> (shift + 8))) continue;
      atomicAdd(&h[wave][(E >> shift) & 255u], (unsigned)Lc.c[i]);
    }
  } else if (mode == SEL_SELECT) {
    const int J = *n_slots;
    const int64_t node_cap = (int64_t)dm.L * dm.G * 2 * dm.N_c;
    const int64_t stride = (int64_t)gridDim.x * 256;
    // Splits: sixteen cost bytes per load (an empty slot or a leaf has cost 0 and
    // its key is never read)
    const int64_t n16 = node_cap / 16;
    for (int64_t v = (int64_t)blockIdx.x * 256 + tid; v < n16; v += stride) {
      const uint4 cw = ((const uint4*)tv.sp_cost)[v];
      if ((cw.x | cw.y | cw.z | cw.w) == 0u) continue;
      const uint32_t wds[4] = {cw.x, cw.y, cw.z, cw.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (wds[q] == 0u) continue;
#pragma unroll
        for (int bt = 0; bt < 4; ++bt) {
          const int c = (wds[q] >> (8 * bt)) & 255u;
          const int64_t i = 16 * v + 4 * q + bt;
          if (c && !(tv.fl_pre_sp && tv.fl_pre_sp[i])) take(tv.sp_E[i], c);
        }
      }
    }
    for (int64_t i = 16 * n16 + (int64_t)blockIdx.x * 256 + tid; i < node_cap; i += stride) {
      const int c = tv.sp_cost[i];
      if (c && !(tv.fl_pre_sp && tv.fl_pre_sp[i])) take(tv.sp_E[i], c);
    }
    // Adds: cost 1 for every unit (l, g, j < J) of the partition
    const int64_t nadd = (int64_t)dm.L * dm.G * J;
    for (int64_t x = (int64_t)blockIdx.x * 256 + tid; x < nadd; x += stride) {
      const int lg = (int)(x / J), j = (int)(x - (int64_t)lg * J);
      const int64_t u = (int64_t)lg * dm.J_cap + j;
      if (!(tv.fl_pre_add && tv.fl_pre_add[u])) take(tv.add_E[u], 1);
    }
    if (pass == 0) {                          // append the workgroup's share to the list
      __syncthreads();
      const unsigned nb = nbuf;
      if (tid == 0)
        lbase = atomicAdd((unsigned long long*)&S->ncand,
                          nb <= SEL_BUF ? (unsigned long long)nb : (unsigned long long)Lc.cap + 1ull);
      __syncthreads();
      if (nb <= SEL_BUF) {
        const uint64_t base = lbase;
        for (unsigned k = tid; k < nb; k += 256) {
          if (base + k < (uint64_t)Lc.cap) { Lc.E[base + k] = bufE[k]; Lc.c[base + k] = bufC[k]; }
        }
      }
    }
  }
  __syncthreads();
  const unsigned hs = h[0][tid] + h[1][tid] + h[2][tid] + h[3][tid];
  if (hs) atomicAdd(&S->hist[tid], (unsigned long long)hs);
  wait_vm();                                  // this thread's histogram atomics are performed
  __syncthreads();
  if (tid == 0) last = atomicAdd(&S->done, 1u) == gridDim.x - 1;
  __syncthreads();
  if (!last) return;
  // the last workgroup: the histogram in one coalesced device-coherent read,
  // cleared for the next pass, then scanned by one thread
  __shared__ unsigned long long hfull[256];
  hfull[tid] = ld_agent(&S->hist[tid]);
  S->hist[tid] = 0;
  __syncthreads();
  if (tid == 0) sel_scan(dm, S, pass, hfull);
}

__global__ __launch_bounds__(256) void k_sel_flag(Dims dm, TreeView tv, const SelState* S) {
  const int32_t* n_slots = tv.nslots;
  const int mode = S->mode;
  const uint64_t theta = S->prefix;
  const int J = *n_slots;
  const int64_t node_cap = (int64_t)dm.L * dm.G * 2 * dm.N_c;
  const int64_t unit_cap = (int64_t)dm.L * dm.G * dm.J_cap;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < node_cap + unit_cap; i += (int64_t)gridDim.x * 256) {
    if (i < node_cap) {
      const int c = tv.sp_cost[i];
      uint8_t x = 0;
      if (c > 0) x = (mode == SEL_ALL) || (mode == SEL_SELECT && tv.sp_E[i] > theta);
      if (tv.fl_pre_sp && tv.fl_pre_sp[i]) x = 1;     // executed by the singleton floor
      tv.sp_exec[i] = x;
    } else {
      const int64_t u = i - node_cap;
      if ((int)(u % dm.J_cap) >= J) continue;
      tv.add_exec[u] = (mode == SEL_ALL) || (mode == SEL_SELECT && tv.add_E[u] > theta) ||
                       (tv.fl_pre_add && tv.fl_pre_add[u]);
    }
  }
}

// Replays the queue rule inside the one group with E == theta.
__global__ void k_sel_group(Dims dm, TreeView tv, SelState* S) {
  const int32_t* n_slots = tv.nslots;
  const int32_t* slot_starts = tv.slots;
  if (threadIdx.x != 0 || S->mode != SEL_SELECT) return;
  const uint64_t theta = S->prefix;
  int64_t R = S->B - S->above;
  const int J = *n_slots;
  const uint32_t id = 0xFFFFFFFFu - (uint32_t)(theta & 0xFFFFFFFFu);
  const uint32_t ord = id >> 8;
  const int lg = (int)(ord / (uint32_t)J), j = (int)(ord % (uint32_t)J);
  const int64_t u = (int64_t)lg * dm.J_cap + j;
  const int64_t base = (int64_t)lg * 2 * dm.N_c + 2 * (int64_t)slot_starts[j];
  // available ops as local indices: 0 = Add, 1 + i = Split(node i)
  int avail[NODE_MAX + 1];
  int na = 0;
  avail[na++] = (int)(id & 255u);
  while (R >= 2 && na > 0) {
    int bi = 0;
    uint64_t bk = 0;
    for (int k = 0; k < na; ++k) {
      const int loc = avail[k];
      const uint64_t key = loc == 0 ? make_key(tv.add_U[u], ord * 256u)
                                    : make_key(tv.sp_U[base + loc - 1], ord * 256u + (uint32_t)loc);
      if (key > bk) { bk = key; bi = k; }
    }
    const int loc = avail[bi];
    avail[bi] = avail[--na];
    int node;
    if (loc == 0) {
      tv.add_exec[u] = 1;
      R -= 1;
      node = 0;                              // Add exposes Split(root)
      if (tv.node_nch[base] > 0 && tv.sp_E[base] == theta) avail[na++] = 1;
    } else {
      node = loc - 1;
      tv.sp_exec[base + node] = 1;
      R -= tv.sp_cost[base + node];
      const int c0 = tv.node_child[base + node], nc = tv.node_nch[base + node];
      for (int k = 0; k < nc; ++k) {
        const int64_t s = base + c0 + k;
        if (tv.node_nch[s] > 0 && tv.sp_E[s] == theta) avail[na++] = 1 + c0 + k;
      }
    }
  }
  S->R = R;
}

// Best available cost-1 op when exactly one unit remains.
__global__ __launch_bounds__(256) void k_sel_resid_find(Dims dm, TreeView tv, SelState* S) {
  const int32_t* n_slots = tv.nslots;
  const int32_t* slot_starts = tv.slots;
  if (!((S->mode == SEL_SELECT || S->mode == SEL_RESID) && S->R == 1)) return;
  const int J = *n_slots;
  uint64_t best = 0;
  // unit by unit: its Add, then the Split slots of its live nodes (the slots
  // of a unit's node range past its live nodes have cost 0); a Split counts
  // if it costs 1, is not executed and its parent's Split (the unit's Add,
  // for the root) is
  const int64_t nu = (int64_t)dm.L * dm.G * J;
  for (int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x; x < nu; x += (int64_t)gridDim.x * 256) {
    const int lg = (int)(x / J), j = (int)(x - (int64_t)lg * J);
    const int64_t u = (int64_t)lg * dm.J_cap + j;
    const uint32_t ord = (uint32_t)lg * (uint32_t)J + (uint32_t)j;
    const bool added = tv.add_exec[u] != 0;
    if (!added) {
      const uint64_t k = make_key(tv.add_U[u], ord * 256u);
      best = k > best ? k : best;
      continue;                               // nothing of the unit's tree is open
    }
    const int64_t base = (int64_t)lg * 2 * dm.N_c + 2 * (int64_t)slot_starts[j];
    const int nn = tv.unit_nn[u];
    for (int loc = 0; loc < nn; ++loc) {
      const int64_t i = base + loc;
      if (tv.sp_cost[i] != 1 || tv.sp_exec[i]) continue;
      const int par = tv.node_parent[i];
      if (par >= 0 && !tv.sp_exec[base + par]) continue;
      const uint64_t k = make_key(tv.sp_U[i], ord * 256u + 1u + (uint32_t)loc);
      best = k > best ? k : best;
    }
  }
  if (best) atomicMax((unsigned long long*)&S->resid_key, (unsigned long long)best);
}

__global__ void k_sel_finish(Dims dm, TreeView tv, SelState* S, int64_t* b_used) {
  const int32_t* n_slots = tv.nslots;
  const int32_t* slot_starts = tv.slots;
  if (threadIdx.x != 0) return;
  const int mode = S->mode;
  int64_t R = S->R;
  if (mode == SEL_ALL) { *b_used = S->floor + S->total; return; }
  if (mode == SEL_NONE) { *b_used = S->floor; return; }
  if (R == 1 && S->resid_key) {
    const int J = *n_slots;
    const uint32_t id = 0xFFFFFFFFu - (uint32_t)(S->resid_key & 0xFFFFFFFFu);
    const uint32_t ord = id >> 8, loc = id & 255u;
    const int lg = (int)(ord / (uint32_t)J), j = (int)(ord % (uint32_t)J);
    if (loc == 0) tv.add_exec[(int64_t)lg * dm.J_cap + j] = 1;
    else tv.sp_exec[(int64_t)lg * 2 * dm.N_c + 2 * (int64_t)slot_starts[j] + loc - 1] = 1;
    R = 0;
  }
  *b_used = S->floor + S->B - R;
}

// ---- the auction with fixed per-(l, g) capacities ---------------------------
// The "w/o Global Allocation" ablation (App. C.3): every (l, g) pair runs the
// queue of the global auction on its own ops with its own capacity
// q_lg = floor(B_free / (L G)) (+1 for the first B_free mod (L G) pairs), and
// budget a pair leaves unused is lost.  One workgroup per pair takes the same
// exact parallel form as the global select: the cost-weighted radix select of
// the cut (the pair's ops read from the tree buffer in each of the eight
// passes), every op above the cut, the group at the cut replayed by one
// thread, and the best available cost-1 op when one unit is left.
__global__ __launch_bounds__(256) void k_sel_pairs(Dims dm, TreeView tv, int64_t* __restrict__ spent) {
  const int lg = blockIdx.x, tid = threadIdx.x, wave = tid >> 6;
  const int J = *tv.nslots;
  const int32_t* slot_starts = tv.slots;
  const int64_t LG = (int64_t)dm.L * dm.G;
  const int64_t Bf = dm.B_free > 0 ? dm.B_free : 0;
  const int64_t q = Bf / LG + (lg < Bf % LG ? 1 : 0);
  const int64_t n0 = (int64_t)lg * 2 * dm.N_c, nn = 2 * dm.N_c;      // the pair's node slots
  const int64_t u0 = (int64_t)lg * dm.J_cap;                         // ... and units j < J
  __shared__ unsigned int h[4][256];
  __shared__ unsigned long long sPrefix;
  __shared__ long long sAbove, sR;
  __shared__ int sMode;
  __shared__ unsigned long long sBest[4];
  if (tid == 0) { sPrefix = 0; sAbove = 0; sMode = SEL_SELECT; sR = 0; }
  // op x of the pair: x < nn a Split slot, else the Add of unit x - nn
  auto op_at = [&](int64_t x, uint64_t& E, int& c) {
    if (x < nn) {
      c = tv.sp_cost[n0 + x];
      E = c ? tv.sp_E[n0 + x] : 0;
    } else {
      c = 1;
      E = tv.add_E[u0 + (x - nn)];
    }
  };
  const int64_t nops = nn + J;
  for (int pass = 0; pass < 8; ++pass) {
#pragma unroll
    for (int w = 0; w < 4; ++w) h[w][tid] = 0;
    __syncthreads();
    const int shift = 56 - 8 * pass;
    const uint64_t pre = sPrefix;
    for (int64_t x = tid; x < nops; x += 256) {
      uint64_t E;
      int c;
      op_at(x, E, c);
      if (!c) continue;
      if (pass > 0 && (E >> (shift + 8)) != (pre >> (shift + 8))) continue;
      atomicAdd(&h[wave][(E >> shift) & 255u], (unsigned)c);
    }
    __syncthreads();
    h[0][tid] += h[1][tid] + h[2][tid] + h[3][tid];
    __syncthreads();
    if (tid == 0) {
      if (pass == 0) {
        int64_t tot = 0;
        for (int k = 0; k < 256; ++k) tot += h[0][k];
        if (q <= 0) sMode = SEL_NONE;
        else if (tot <= q) { sMode = SEL_ALL; sR = q - tot; }
        else if (q == 1) { sMode = SEL_RESID; sR = 1; }
      }
      if (sMode == SEL_SELECT) {
        const int64_t need = (q - 1) - sAbove;     // the cut's rank q - 1 within the pair
        int64_t cum = 0;
        for (int k = 255; k >= 0; --k) {
          const int64_t hk = h[0][k];
          if (cum + hk >= need) { sPrefix |= (uint64_t)k << shift; sAbove += cum; break; }
          cum += hk;
        }
      }
    }
    __syncthreads();
    if (sMode != SEL_SELECT) break;
  }
  const int mode = sMode;
  const uint64_t theta = sPrefix;
  // every op above the cut (all of them when the pair's ops fit its capacity)
  for (int64_t x = tid; x < nops; x += 256) {
    uint64_t E;
    int c;
    op_at(x, E, c);
    const uint8_t ex = c > 0 && (mode == SEL_ALL || (mode == SEL_SELECT && E > theta));
    if (x < nn) tv.sp_exec[n0 + x] = ex; else tv.add_exec[u0 + (x - nn)] = ex;
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");   // the flags, visible to the workgroup
  __syncthreads();
  if (tid == 0 && mode == SEL_SELECT) {
    // the group at the cut lies in one unit of this pair: the queue rule replayed there
    int64_t R = q - sAbove;
    const uint32_t id = 0xFFFFFFFFu - (uint32_t)(theta & 0xFFFFFFFFu);
    const uint32_t ord = id >> 8;
    const int j = (int)(ord % (uint32_t)J);
    const int64_t u = u0 + j;
    const int64_t base = n0 + 2 * (int64_t)slot_starts[j];
    int avail[NODE_MAX + 1];
    int na = 0;
    avail[na++] = (int)(id & 255u);
    while (R >= 2 && na > 0) {
      int bi = 0;
      uint64_t bk = 0;
      for (int k = 0; k < na; ++k) {
        const int loc = avail[k];
        const uint64_t key = loc == 0 ? make_key(tv.add_U[u], ord * 256u)
                                      : make_key(tv.sp_U[base + loc - 1], ord * 256u + (uint32_t)loc);
        if (key > bk) { bk = key; bi = k; }
      }
      const int loc = avail[bi];
      avail[bi] = avail[--na];
      if (loc == 0) {
        tv.add_exec[u] = 1;
        R -= 1;
        if (tv.node_nch[base] > 0 && tv.sp_E[base] == theta) avail[na++] = 1;
      } else {
        const int node = loc - 1;
        tv.sp_exec[base + node] = 1;
        R -= tv.sp_cost[base + node];
        const int c0 = tv.node_child[base + node], nc = tv.node_nch[base + node];
        for (int k = 0; k < nc; ++k) {
          const int64_t sl = base + c0 + k;
          if (tv.node_nch[sl] > 0 && tv.sp_E[sl] == theta) avail[na++] = 1 + c0 + k;
        }
      }
    }
    sR = R;
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  __syncthreads();
  if (sR == 1 && mode != SEL_ALL && mode != SEL_NONE) {
    // one unit left: the best available cost-1 op of the pair (its creating op executed, itself not)
    uint64_t best = 0;
    for (int64_t x = tid; x < nops; x += 256) {
      if (x < nn) {
        const int64_t i = n0 + x;
        if (tv.sp_cost[i] != 1 || tv.sp_exec[i]) continue;
        const int o = (int)x;
        int lo = 0, hi = J - 1;                  // unit j with 2 a_j <= o < 2 a_{j+1}
        while (lo < hi) {
          const int mid = (lo + hi + 1) >> 1;
          if (2 * slot_starts[mid] <= o) lo = mid; else hi = mid - 1;
        }
        const int64_t base = n0 + 2 * (int64_t)slot_starts[lo];
        const int par = tv.node_parent[i];
        const bool pe = par < 0 ? tv.add_exec[u0 + lo] : tv.sp_exec[base + par];
        if (!pe) continue;
        const uint32_t ord = (uint32_t)lg * (uint32_t)J + (uint32_t)lo;
        const uint64_t k = make_key(tv.sp_U[i], ord * 256u + 1u + (uint32_t)(i - base));
        best = k > best ? k : best;
      } else {
        const int j = (int)(x - nn);
        if (tv.add_exec[u0 + j]) continue;
        const uint32_t ord = (uint32_t)lg * (uint32_t)J + (uint32_t)j;
        const uint64_t k = make_key(tv.add_U[u0 + j], ord * 256u);
        best = k > best ? k : best;
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const uint64_t b2 = __shfl_xor(best, o, 64);
      best = b2 > best ? b2 : best;
    }
    if ((tid & 63) == 0) sBest[wave] = best;
    __syncthreads();
    if (tid == 0) {
      uint64_t b = sBest[0];
      for (int w = 1; w < 4; ++w) b = sBest[w] > b ? sBest[w] : b;
      if (b) {
        const uint32_t id = 0xFFFFFFFFu - (uint32_t)(b & 0xFFFFFFFFu);
        const uint32_t ord = id >> 8, loc = id & 255u;
        const int j = (int)(ord % (uint32_t)J);
        if (loc == 0) tv.add_exec[u0 + j] = 1;
        else tv.sp_exec[n0 + 2 * (int64_t)slot_starts[j] + loc - 1] = 1;
        sR = 0;
      }
    }
  }
  __syncthreads();
  if (tid == 0) spent[lg] = mode == SEL_NONE ? 0 : q - sR;
}

__global__ void k_sel_pairs_sum(Dims dm, const int64_t* __restrict__ spent, int64_t* b_used) {
  if (threadIdx.x != 0) return;
  int64_t s = 0;
  for (int64_t i = 0; i < (int64_t)dm.L * dm.G; ++i) s += spent[i];
  *b_used = s;
}

// the eight radix passes of one cost-weighted select
static void sel_passes(const Dims& dm, const TreeView& tv, SelState* S, hipStream_t st) {
  const int64_t tot = sel_ops(dm);
  const unsigned blocks = (unsigned)std::min<int64_t>((tot + 255) / 256, SEL_GRID);
  const SelList Lc = sel_list(S, dm);
  for (int pass = 0; pass < 8; ++pass) {
    // few workgroups: their per-pass global atomics (list base, histogram, completion) meet at single
    // addresses
    const unsigned g = std::min<unsigned>(blocks, pass == 0 ? 512u : 256u);
    hipLaunchKernelGGL(k_sel_hist, dim3(g), dim3(256), 0, st, dm, tv, S, pass, Lc);
  }
}

hipError_t launch_select(const Dims& dm, const TreeView& tv, int64_t* b_used, void* ws, hipStream_t st) {
  if (dm.pair_quotas) {
    int64_t* spent = (int64_t*)ws;            // [L*G] spent per pair
    hipLaunchKernelGGL(k_sel_pairs, dim3((unsigned)(dm.L * dm.G)), dim3(256), 0, st, dm, tv, spent);
    hipLaunchKernelGGL(k_sel_pairs_sum, dim3(1), dim3(64), 0, st, dm, (const int64_t*)spent, b_used);
    return hipGetLastError();
  }
  SelState* S = (SelState*)ws;
  hipLaunchKernelGGL(k_sel_init, dim3(1), dim3(256), 0, st, dm, S, 0, tv.fl_state);
  const int64_t tot = (int64_t)dm.L * dm.G * 2 * dm.N_c + (int64_t)dm.L * dm.G * dm.J_cap;
  const unsigned blocks = (unsigned)std::min<int64_t>((tot + 255) / 256, 4096);
  sel_passes(dm, tv, S, st);
  hipLaunchKernelGGL(k_sel_flag, dim3(blocks), dim3(256), 0, st, dm, tv, (const SelState*)S);
  hipLaunchKernelGGL(k_sel_group, dim3(1), dim3(64), 0, st, dm, tv, S);
  hipLaunchKernelGGL(k_sel_resid_find, dim3(blocks), dim3(256), 0, st, dm, tv, S);
  hipLaunchKernelGGL(k_sel_finish, dim3(1), dim3(64), 0, st, dm, tv, S, b_used);
  return hipGetLastError();
}

// Lower bound of the cut over the ops known so far (the pruned build): the
// same cost-weighted radix select; with every known op affordable nothing can
// be pruned (bound 0); with B_free <= 1 no Split can execute (bound max).
__global__ void k_theta_store(Dims dm, const SelState* S, uint64_t* theta, bool skip_bound) {
  if (threadIdx.x != 0) return;
  const int mode = S->mode;
  const uint64_t v = mode == SEL_SELECT ? S->prefix : (mode == SEL_ALL ? 0ull : ~0ull);
  theta[0] = v;
  if (skip_bound) theta[1] = v;
}

hipError_t launch_theta(const Dims& dm, const TreeView& tv, hipStream_t st, bool skip_bound) {
  SelState* S = (SelState*)tv.selstate;
  hipLaunchKernelGGL(k_sel_init, dim3(1), dim3(256), 0, st, dm, S, skip_bound ? 1 : 0, (const int64_t*)nullptr);
  sel_passes(dm, tv, S, st);
  hipLaunchKernelGGL(k_theta_store, dim3(1), dim3(64), 0, st, dm, (const SelState*)S, tv.theta, skip_bound);
  return hipGetLastError();
}

}  // namespace gkv
