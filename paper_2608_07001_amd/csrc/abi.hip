// Host side of the C ABI: defaults, size planning, argument validation and
// the five entry points.  Every entry point validates on the host and only
// enqueues kernels on the caller's stream.
#include <math.h>
#include <string.h>

#include <mutex>
#include <vector>

#include "common.h"

using namespace gkv;

namespace gkv {

static size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

Dims make_dims(const gracekv_config& c, const gracekv_plan& p) {
  Dims d;
  memset(&d, 0, sizeof(d));
  d.L = c.L; d.G = c.G; d.H = c.H; d.d = c.d; d.hpg = c.H / c.G; d.W = c.W; d.n_seg = c.n_seg;
  d.Dh = c.D_hidden; d.dtype = c.dtype; d.r = p.r; d.J_cap = p.J_cap;
  d.T = p.T; d.N_ctx = c.N_ctx; d.N_c = p.N_c; d.B_total = p.B_total; d.B_free = p.B_free;
  d.lam_stab = c.lam_stab; d.lam_s = c.lam_s; d.eps_seg = c.eps_seg; d.mad = c.mad_factor;
  d.win[0] = c.win[0]; d.win[1] = c.win[1]; d.win[2] = c.win[2];
  d.n_min = c.n_min; d.n_max = c.n_max; d.n0 = c.n0;
  d.lam_d = c.lam_d; d.lam_n = c.lam_n; d.c_cut = c.c_cut;
  d.lam_Z = c.lam_Z; d.lam_M = c.lam_M; d.lam_kappa = c.lam_kappa; d.beta_frac = c.beta_frac; d.eps = c.eps;
  d.k_curv = c.k_curv;
  d.rows = d.hpg * c.W;
  d.dp_serial = (c.flags & GRACEKV_FLAG_DP_SERIAL) ? 1 : 0;
  d.uniform_slots = (c.flags & GRACEKV_FLAG_UNIFORM_SLOTS) ? 1 : 0;
  d.pair_quotas = (c.flags & GRACEKV_FLAG_PAIR_QUOTAS) ? 1 : 0;
  d.lam_graph = c.lambda_graph;
  d.stage_times = (c.flags & GRACEKV_FLAG_STAGE_TIMES) ? 1 : 0;
  d.alpha_floor = (float)c.alpha_floor;
  d.floor_cap = c.alpha_floor > 0.0 ? (int64_t)floor(c.alpha_floor * (double)p.B_free) : 0;
  // propagation layers at relative depths 0.50 and 0.75, rounded like the
  // segmentation layers (eq:app_seg_layers)
  d.n_gl = 0;
  const int cand[2] = {c.L / 2, (3 * c.L) / 4};
  for (int i = 0; i < 2; ++i) {
    const int l = cand[i] < c.L - 1 ? cand[i] : c.L - 1;
    if (d.n_gl == 0 || d.gl[0] != l) d.gl[d.n_gl++] = l;
  }
  return d;
}

TreeView make_view(void* base, const gracekv_plan& p) {
  char* b = (char*)base;
  TreeView v;
  v.node_a = (int32_t*)(b + p.off_node_a);
  v.node_n = (int32_t*)(b + p.off_node_n);
  v.node_child = (int32_t*)(b + p.off_node_child);
  v.node_parent = (int32_t*)(b + p.off_node_parent);
  v.node_nch = (uint8_t*)(b + p.off_node_nch);
  v.node_kind = (uint8_t*)(b + p.off_node_kind);
  v.node_cut = (int32_t*)(b + p.off_node_cut);
  v.node_D = (float*)(b + p.off_node_D);
  v.node_R = (float*)(b + p.off_node_R);
  v.sp_U = (float*)(b + p.off_sp_U);
  v.sp_E = (uint64_t*)(b + p.off_sp_E);
  v.sp_cost = (uint8_t*)(b + p.off_sp_cost);
  v.sp_exec = (uint8_t*)(b + p.off_sp_exec);
  v.unit_nn = (int32_t*)(b + p.off_unit_nn);
  v.unit_Ddrop = (float*)(b + p.off_unit_Ddrop);
  v.add_U = (float*)(b + p.off_add_U);
  v.add_E = (uint64_t*)(b + p.off_add_E);
  v.add_exec = (uint8_t*)(b + p.off_add_exec);
  v.tok_R = (float*)(b + p.off_tok_R);
  v.tok_A = (float*)(b + p.off_tok_A);
  v.row_stats = (float4*)(b + p.off_row_stats);
  v.probe_m = (float*)(b + p.off_probe_m);
  v.probe_ZC = (float*)(b + p.off_probe_ZC);
  v.lg_S = (float*)(b + p.off_lg_S);
  v.omega = (float*)(b + p.off_omega);
  v.status = (int32_t*)(b + p.off_status);
  v.slots = (int32_t*)(b + p.off_slots);
  v.proto = (void*)(b + p.off_proto);
  v.proto_logm = (float*)(b + p.off_proto_logm);
  v.kargs = (void*)(b + p.tree_bytes - KARGS_BYTES);
  v.nslots = (int32_t*)(b + p.off_nslots);
  v.theta = (uint64_t*)(b + p.off_theta);
  v.selstate = (void*)(b + p.off_selstate);
  v.work = (int32_t*)(b + p.off_work);
  v.wctr = (int32_t*)(b + p.off_wctr);
  v.dhat = nullptr;
  v.fl_flag = nullptr;
  v.fl_pre_add = nullptr;
  v.fl_pre_sp = nullptr;
  v.fl_state = nullptr;
  // the level region sits just before the kernel-argument copy
  const int64_t LG = p.unit_cap / p.J_cap;
  char* lv = b + p.tree_bytes - KARGS_BYTES - level_region_bytes(LG, p.N_c, p.unit_cap);
  const int64_t cap = level_capacity(LG, p.N_c);
  size_t o = 0;
  auto take = [&](size_t bytes) { char* q = lv + o; o = (o + bytes + 255) & ~(size_t)255; return q; };
  v.lv_items = (int32_t*)take((size_t)cap * 32);
  v.lv_res = (int32_t*)take((size_t)cap * 48);
  v.lv_units = (int32_t*)take((size_t)p.unit_cap * 8);
  v.lv_state = (int4*)take((size_t)p.unit_cap * 16);
  v.lv_ctr = (int32_t*)take(64);
  v.lv_cap = cap;
  return v;
}

// the floor's region (alpha_floor > 0) and the view's pointers into it
static FloorView floor_of(void* trees, const Dims& dm, const gracekv_plan& p, TreeView* tv) {
  FloorView f = floor_view((char*)trees + p.off_floor, dm, p.unit_cap, p.node_cap);
  if (tv) {
    tv->fl_flag = f.flag;
    tv->fl_pre_add = f.pre_add;
    tv->fl_pre_sp = f.pre_sp;
    tv->fl_state = f.state;
  }
  return f;
}

__global__ void k_copy_slots(const int32_t* __restrict__ slot_starts, const int32_t* __restrict__ n_slots, int J_cap,
                             TreeView tv) {
  for (int i = threadIdx.x; i <= J_cap; i += blockDim.x) tv.slots[i] = slot_starts[i];
  // the status word is cleared and the buffer marked as built before any
  // later kernel of the build can latch a fault into it
  if (threadIdx.x == 0) { *tv.nslots = *n_slots; tv.status[0] = 0; tv.status[1] = STATUS_BUILT; }
}

// Copies the kernel arguments into the tree buffer, in stream order, for the
// kernels that read them through pointers (their argument structures would not
// fit in scalar registers).
__global__ void k_store_args(Dims dm, TreeView tv) {
  if (threadIdx.x == 0) {
    *(Dims*)tv.kargs = dm;
    *(TreeView*)((char*)tv.kargs + 512) = tv;
  }
}

hipError_t launch_store_args(const Dims& dm, const TreeView& tv, hipStream_t st) {
  static_assert(sizeof(Dims) <= 512 && sizeof(TreeView) <= KARGS_BYTES - 512, "kernel argument copy too small");
  hipLaunchKernelGGL(k_store_args, dim3(1), dim3(64), 0, st, dm, tv);
  return hipGetLastError();
}


// ---- stage clock ----
// Event pairs recorded by calls with GRACEKV_FLAG_STAGE_TIMES wait in `pending`
// until gracekv_stage_times reads them; read events go back to a per-device pool.
namespace {
struct ClockPair { int stage, device; hipEvent_t a, b; };
std::mutex clock_mu;
std::vector<ClockPair> clock_pending;
std::vector<std::pair<int, hipEvent_t>> clock_pool;

hipEvent_t clock_event(int dev) {
  for (size_t i = 0; i < clock_pool.size(); ++i)
    if (clock_pool[i].first == dev) {
      hipEvent_t e = clock_pool[i].second;
      clock_pool[i] = clock_pool.back();
      clock_pool.pop_back();
      return e;
    }
  hipEvent_t e = nullptr;
  return hipEventCreate(&e) == hipSuccess ? e : nullptr;
}
}  // namespace

int clock_begin(const Dims& dm, int stage, hipStream_t st) {
  if (!dm.stage_times) return -1;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  std::lock_guard<std::mutex> g(clock_mu);
  hipEvent_t a = clock_event(dev), b = clock_event(dev);
  if (!a || !b || hipEventRecord(a, st) != hipSuccess) {
    if (a) clock_pool.push_back({dev, a});
    if (b) clock_pool.push_back({dev, b});
    return -1;
  }
  clock_pending.push_back({stage, dev, a, b});
  return (int)clock_pending.size() - 1;
}

void clock_end(int handle, hipStream_t st) {
  if (handle < 0) return;
  std::lock_guard<std::mutex> g(clock_mu);
  if (handle < (int)clock_pending.size() && hipEventRecord(clock_pending[handle].b, st) != hipSuccess) {
    clock_pool.push_back({clock_pending[handle].device, clock_pending[handle].b});
    clock_pending[handle].b = nullptr;
  }
}

}  // namespace gkv

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

extern "C" {

int32_t gracekv_abi_version(void) { return GRACEKV_ABI_VERSION; }

gracekv_status gracekv_default_config(gracekv_config* c) {
  if (!c) return GRACEKV_ERR_INVALID_ARG;
  memset(c, 0, sizeof(*c));
  c->n_seg = 3;
  c->dtype = GRACEKV_BF16;
  c->x = 1.0;
  c->r_default = 32; c->r_min = 4;
  c->lam_stab = 0.25f; c->lam_s = 0.15f; c->eps_seg = 1e-6f; c->mad_factor = 1.4826f;
  c->win[0] = 4; c->win[1] = 8; c->win[2] = 16;
  c->n_min = 16; c->n_max = 128; c->n0 = 64;
  c->lam_d = 0.25f; c->lam_n = 0.10f; c->c_cut = 1.0f;
  c->lam_Z = 0.25f; c->lam_M = 0.75f;
  c->k_curv = 16;
  c->lam_kappa = 0.05f; c->beta_frac = 0.1f; c->eps = 1e-6f;
  c->lambda_graph = 0.f; c->alpha_floor = 0.0;
  return GRACEKV_OK;
}

const char* gracekv_status_string(gracekv_status s) {
  switch (s) {
    case GRACEKV_OK: return "ok";
    case GRACEKV_ERR_INVALID_ARG: return "invalid argument";
    case GRACEKV_ERR_UNSUPPORTED: return "unsupported configuration";
    case GRACEKV_ERR_BUDGET: return "budget cannot hold the minimum recent window";
    case GRACEKV_ERR_WORKSPACE: return "workspace too small";
    case GRACEKV_ERR_HIP: return "HIP error";
    case GRACEKV_ERR_NUMERIC: return "non-finite gain on the device";
    case GRACEKV_ERR_STATE: return "the tree buffer holds no build";
    case GRACEKV_ERR_PARTITION: return "malformed slot partition on the device";
    case GRACEKV_ERR_CAPACITY: return "packed cache over its capacity on the device";
  }
  return "unknown status";
}

gracekv_status gracekv_plan_sizes(const gracekv_config* c, gracekv_plan* p) {
  if (!c || !p) return GRACEKV_ERR_INVALID_ARG;
  memset(p, 0, sizeof(*p));
  if (c->L < 1 || c->G < 1 || c->H < 1 || c->d < 2 || c->W < 1 || c->N_ctx < 1 || c->n_seg < 1 || c->D_hidden < 1)
    return GRACEKV_ERR_INVALID_ARG;
  if (c->H % c->G != 0) return GRACEKV_ERR_INVALID_ARG;
  if (c->dtype != GRACEKV_F32 && c->dtype != GRACEKV_BF16) return GRACEKV_ERR_INVALID_ARG;
  if (!(c->x >= 1.0) || !isfinite(c->x)) return GRACEKV_ERR_INVALID_ARG;
  if (!(c->lambda_graph >= 0.f && c->lambda_graph <= 1.f)) return GRACEKV_ERR_INVALID_ARG;
  if (c->lambda_graph > 0.f && c->H / c->G > 8) return GRACEKV_ERR_UNSUPPORTED;   // one wave per query head
  if (!(c->alpha_floor >= 0.0 && c->alpha_floor <= 1.0)) return GRACEKV_ERR_INVALID_ARG;
  if (c->alpha_floor > 0.0 && (c->flags & (GRACEKV_FLAG_PRUNE | GRACEKV_FLAG_PAIR_QUOTAS)))
    return GRACEKV_ERR_UNSUPPORTED;   // the floor needs every tree complete and the shared auction
  if (c->flags & ~(GRACEKV_FLAG_PRUNE | GRACEKV_FLAG_DP_SERIAL | GRACEKV_FLAG_UNIFORM_SLOTS |
                   GRACEKV_FLAG_PAIR_QUOTAS | GRACEKV_FLAG_STATS_READY | GRACEKV_FLAG_STAGE_TIMES))
    return GRACEKV_ERR_INVALID_ARG;
  // the pruning bounds are those of the shared auction
  if ((c->flags & GRACEKV_FLAG_PAIR_QUOTAS) && (c->flags & GRACEKV_FLAG_PRUNE)) return GRACEKV_ERR_UNSUPPORTED;
  if (c->d != 64 && c->d != 128) return GRACEKV_ERR_UNSUPPORTED;
  if (c->dtype == GRACEKV_F32 && c->d != 64) return GRACEKV_ERR_UNSUPPORTED;   // refinement LDS
  if (c->D_hidden % 8 != 0) return GRACEKV_ERR_UNSUPPORTED;                   // 16-byte hidden rows
  if (c->W > WMAX || c->n_seg > 8) return GRACEKV_ERR_UNSUPPORTED;
  if (c->n_min < 16 || c->n_max > NMAX || c->n_max < c->n_min || c->n0 < 1) return GRACEKV_ERR_UNSUPPORTED;
  if (c->win[0] != 4 || c->win[1] != 8 || c->win[2] != 16) return GRACEKV_ERR_UNSUPPORTED;
  if (c->k_curv < 0 || c->k_curv > CAND_MAX - 2) return GRACEKV_ERR_UNSUPPORTED;
  // uniform slots: J = ceil(N_c / n0) stays within the slot capacity floor(N_c / n_min) + 1
  if ((c->flags & GRACEKV_FLAG_UNIFORM_SLOTS) && (c->n0 > c->n_max || c->n0 < c->n_min))
    return GRACEKV_ERR_UNSUPPORTED;
  const int64_t T = c->N_ctx + c->W;
  if (T > (int64_t)0x7fffffff / 2) return GRACEKV_ERR_UNSUPPORTED;
  const int64_t LG = (int64_t)c->L * c->G;
  const int64_t B_total = (int64_t)floor((double)LG * (double)c->N_ctx / c->x);
  int64_t r = c->r_default;
  if (LG * r > B_total) r = B_total / LG;
  if (r > c->N_ctx) r = c->N_ctx;
  if (r < c->r_min) return GRACEKV_ERR_BUDGET;
  p->T = T;
  p->r = (int32_t)r;
  p->N_c = c->N_ctx - r;
  p->B_total = B_total;
  p->B_free = B_total - LG * r;
  p->J_cap = (int32_t)(p->N_c / c->n_min + 1);
  p->unit_cap = LG * p->J_cap;
  p->node_cap = LG * 2 * p->N_c;
  gracekv_plan tmp = *p;
  Dims dm = make_dims(*c, tmp);
  p->build_lds_bytes = build_lds_bytes(dm);
  if (p->build_lds_bytes > 160 * 1024 || root_lds_bytes(dm) > 160 * 1024 || split_root_lds_bytes(c->d) > 80 * 1024)
    return GRACEKV_ERR_UNSUPPORTED;
  const size_t NC = (size_t)p->node_cap, UC = (size_t)p->unit_cap;
  size_t o = 0;
  auto put = [&](size_t& off, size_t bytes) { off = o; o = al256(o + bytes); };
  put(p->off_sp_E, NC * 8);
  put(p->off_add_E, UC * 8);
  put(p->off_node_a, NC * 4);
  put(p->off_node_n, NC * 4);
  put(p->off_node_child, NC * 4);
  put(p->off_node_parent, NC * 4);
  put(p->off_node_cut, NC * 4);
  put(p->off_node_D, NC * 4);
  put(p->off_node_R, NC * 4);
  put(p->off_sp_U, NC * 4);
  put(p->off_node_nch, NC);
  put(p->off_node_kind, NC);
  put(p->off_sp_cost, NC);
  put(p->off_sp_exec, NC);
  put(p->off_unit_nn, UC * 4);
  put(p->off_unit_Ddrop, UC * 4);
  put(p->off_add_U, UC * 4);
  put(p->off_add_exec, UC);
  put(p->off_tok_R, (size_t)LG * p->N_c * 4);
  put(p->off_tok_A, (size_t)LG * p->N_c * 4);
  put(p->off_row_stats, (size_t)LG * dm.rows * 16);
  put(p->off_probe_m, (size_t)LG * c->W * 4);
  put(p->off_probe_ZC, (size_t)LG * c->W * 4);
  put(p->off_lg_S, (size_t)LG * 4);
  put(p->off_omega, (size_t)LG * 4);
  put(p->off_status, 16);
  put(p->off_slots, (size_t)(p->J_cap + 1) * 4);
  put(p->off_nslots, 16);
  put(p->off_partial, (size_t)LG * rowstats_chunks(dm) * dm.rows * 16);
  put(p->off_theta, 16);
  put(p->off_selstate, selstate_bytes(dm));
  put(p->off_work, UC * 32);                // work items: 8 int32 each
  put(p->off_wctr, 16);
  put(p->off_proto, UC * 2 * (size_t)c->d * (c->dtype == GRACEKV_BF16 ? 2 : 4));
  put(p->off_proto_logm, UC * 4);
  put(p->off_floor, c->alpha_floor > 0.0 ? floor_view(nullptr, dm, p->unit_cap, p->node_cap).bytes : 0);
  o += level_region_bytes(LG, p->N_c, p->unit_cap);   // level-by-level refinement lists
  o += KARGS_BYTES;                          // device copy of the kernel arguments
  p->tree_bytes = o;
  p->seg_ws_bytes = segment_ws_bytes(dm);
  p->sel_ws_bytes = select_ws_bytes(dm);
  p->pack_ws_bytes = pack_ws_bytes(dm);
  p->build_ws_bytes = mh_bytes(dm);
  return GRACEKV_OK;
}

static gracekv_status prep(const gracekv_config* c, gracekv_plan* p) {
  if (!c) return GRACEKV_ERR_INVALID_ARG;
  return gracekv_plan_sizes(c, p);
}

static gracekv_status hip_status(hipError_t e) { return e == hipSuccess ? GRACEKV_OK : GRACEKV_ERR_HIP; }

gracekv_status gracekv_check(const gracekv_config* c, void* trees, void* stream) {
  gracekv_plan p;
  gracekv_status s = prep(c, &p);
  if (s != GRACEKV_OK) return s;
  if (!trees) return GRACEKV_ERR_INVALID_ARG;
  if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return GRACEKV_ERR_HIP;
  int32_t st[2] = {0, 0};
  if (hipMemcpy(st, (char*)trees + p.off_status, 8, hipMemcpyDeviceToHost) != hipSuccess) return GRACEKV_ERR_HIP;
  if (st[1] != STATUS_BUILT) return GRACEKV_ERR_STATE;
  if (st[0] & STATUS_NUMERIC) return GRACEKV_ERR_NUMERIC;
  if (st[0] & STATUS_PARTITION) return GRACEKV_ERR_PARTITION;
  if (st[0] & STATUS_CAPACITY) return GRACEKV_ERR_CAPACITY;
  return GRACEKV_OK;
}

gracekv_status gracekv_segment(const gracekv_config* c, const void* hidden, const float* surprisal, float* kappa,
                               float* bscore, int32_t* slot_starts, int32_t* n_slots, void* ws, size_t ws_bytes,
                               void* stream) {
  gracekv_plan p;
  gracekv_status s = prep(c, &p);
  if (s != GRACEKV_OK) return s;
  if (!hidden || !surprisal || !kappa || !bscore || !slot_starts || !n_slots || !ws) return GRACEKV_ERR_INVALID_ARG;
  if (!aligned16(hidden) || !aligned16(ws)) return GRACEKV_ERR_INVALID_ARG;
  if (ws_bytes < p.seg_ws_bytes) return GRACEKV_ERR_WORKSPACE;
  Dims dm = make_dims(*c, p);
  const int clk = clock_begin(dm, GRACEKV_STAGE_SEGMENT, (hipStream_t)stream);
  const hipError_t e = launch_segment(dm, hidden, surprisal, kappa, bscore, slot_starts, n_slots, ws, (hipStream_t)stream);
  clock_end(clk, (hipStream_t)stream);
  return hip_status(e);
}

gracekv_status gracekv_stage_times(float* total_ms, int32_t* launches) {
  if (!total_ms || !launches) return GRACEKV_ERR_INVALID_ARG;
  for (int i = 0; i < GRACEKV_N_STAGES; ++i) { total_ms[i] = 0.f; launches[i] = 0; }
  std::lock_guard<std::mutex> g(clock_mu);
  gracekv_status s = GRACEKV_OK;
  int cur = -1;
  (void)hipGetDevice(&cur);
  for (const ClockPair& p : clock_pending) {
    if (p.b && p.stage >= 0 && p.stage < GRACEKV_N_STAGES && s == GRACEKV_OK) {
      float ms = 0.f;
      (void)hipSetDevice(p.device);
      if (hipEventSynchronize(p.b) != hipSuccess || hipEventElapsedTime(&ms, p.a, p.b) != hipSuccess) {
        s = GRACEKV_ERR_HIP;
      } else {
        total_ms[p.stage] += ms;
        launches[p.stage] += 1;
      }
    }
    clock_pool.push_back({p.device, p.a});
    if (p.b) clock_pool.push_back({p.device, p.b});
  }
  clock_pending.clear();
  if (cur >= 0) (void)hipSetDevice(cur);
  return s;
}

gracekv_status gracekv_build_trees(const gracekv_config* c, const void* K, const void* V, const void* Q,
                                   const void* Q_graph, const float* rope_cos, const float* rope_sin,
                                   const int32_t* slot_starts, const int32_t* n_slots, const float* kappa,
                                   const float* omega_raw, void* trees, void* ws, size_t ws_bytes, void* stream) {
  gracekv_plan p;
  gracekv_status s = prep(c, &p);
  if (s != GRACEKV_OK) return s;
  if (!K || !V || !Q || !rope_cos || !rope_sin || !slot_starts || !n_slots || !kappa || !trees)
    return GRACEKV_ERR_INVALID_ARG;
  if (!aligned16(K) || !aligned16(V) || !aligned16(Q) || !aligned16(trees)) return GRACEKV_ERR_INVALID_ARG;
  const bool graph = c->lambda_graph > 0.f;
  if (graph) {
    if (!Q_graph || !ws || !aligned16(Q_graph) || !aligned16(ws)) return GRACEKV_ERR_INVALID_ARG;
    if (ws_bytes < p.build_ws_bytes) return GRACEKV_ERR_WORKSPACE;
  }
  Dims dm = make_dims(*c, p);
  TreeView tv = make_view(trees, p);
  FloorView fv{};
  if (c->alpha_floor > 0.0) fv = floor_of(trees, dm, p, &tv);
  hipStream_t st = (hipStream_t)stream;
  hipLaunchKernelGGL(k_copy_slots, dim3(1), dim3(256), 0, st, slot_starts, n_slots, p.J_cap, tv);
  if (hipGetLastError() != hipSuccess) return GRACEKV_ERR_HIP;
  if (launch_store_args(dm, tv, st) != hipSuccess) return GRACEKV_ERR_HIP;
  if (!(c->flags & GRACEKV_FLAG_STATS_READY)) {
    const int clk = clock_begin(dm, GRACEKV_STAGE_ROWSTATS, st);
    const hipError_t e = launch_rowstats(dm, K, Q, tv, (float4*)((char*)trees + p.off_partial), st);
    clock_end(clk, st);
    if (e != hipSuccess) return GRACEKV_ERR_HIP;
  }
  if (token_relevance_pass(dm)) {
    const int clk = clock_begin(dm, GRACEKV_STAGE_TOKEN_RELEVANCE, st);
    const hipError_t e = launch_token_relevance(dm, K, Q, tv, st);
    clock_end(clk, st);
    if (e != hipSuccess) return GRACEKV_ERR_HIP;
  }
  // one clock pair per stage: the root splits, then everything below them (the
  // depths refined level by level and the per-unit kernel after them)
  auto build = [&](int mode) {
    const bool roots = mode == BUILD_ROOT_SPLIT || mode == BUILD_ROOT_FULL;
    const int clk = clock_begin(dm, roots ? GRACEKV_STAGE_ROOT_SPLIT : GRACEKV_STAGE_REFINE, st);
    hipError_t e = hipSuccess;
    const bool levels = !roots && dm.dtype == GRACEKV_BF16;
    if (levels)
      e = launch_levels_bf16(dm, mode == BUILD_FULL, K, V, Q, rope_cos, rope_sin, slot_starts, n_slots, kappa, tv, st);
    if (e == hipSuccess)
      e = launch_build(dm, p.build_lds_bytes, mode, K, V, Q, rope_cos, rope_sin, slot_starts, n_slots, kappa, tv, st,
                       levels);
    clock_end(clk, st);
    return e;
  };
  if (launch_omega(dm, omega_raw, tv, st) != hipSuccess) return GRACEKV_ERR_HIP;
  // multi-hop relevance: s-hat of every (l, g) first (bf16: the token relevance
  // pass above; fp32: a root pass without the mix), then seeds and hops, then
  // the roots with R^tok = (1 - lambda) s-hat + lambda d-hat
  const bool graph_first = graph && token_relevance_pass(dm);
  if (graph && !graph_first &&
      launch_root(dm, K, V, Q, rope_cos, rope_sin, slot_starts, n_slots, tv, st) != hipSuccess)
    return GRACEKV_ERR_HIP;
  if (graph) {
    if (launch_multihop(dm, K, Q, Q_graph, tv, ws, st) != hipSuccess) return GRACEKV_ERR_HIP;
    tv.dhat = mh_view(ws, dm).dhat;
    if (launch_store_args(dm, tv, st) != hipSuccess) return GRACEKV_ERR_HIP;
  }
  {
    const int clk = clock_begin(dm, GRACEKV_STAGE_ROOT, st);
    const hipError_t e = launch_root(dm, K, V, Q, rope_cos, rope_sin, slot_starts, n_slots, tv, st);
    clock_end(clk, st);
    if (e != hipSuccess) return GRACEKV_ERR_HIP;
  }
  // singleton floor: the candidates, from the final token values, before any split
  if (c->alpha_floor > 0.0) {
    const int clk = clock_begin(dm, GRACEKV_STAGE_FLOOR_CANDIDATES, st);
    const hipError_t e = launch_floor_candidates(dm, tv, fv, st);
    clock_end(clk, st);
    if (e != hipSuccess) return GRACEKV_ERR_HIP;
  }
  if (!(c->flags & GRACEKV_FLAG_PRUNE)) {
    // bf16: the roots first, by the kernel the pruned build refines them with
    if (c->dtype == GRACEKV_BF16 && build(BUILD_ROOT_FULL) != hipSuccess) return GRACEKV_ERR_HIP;
    return hip_status(build(BUILD_FULL));
  }
  // pruned: bound from the roots -> root splits -> tighter bound -> the rest.  The
  // first bound is taken at rank B_free (one below the cut's rank B_free - 1): it
  // is still a lower bound of the cut, and at least one Add keyed at or above it
  // is left unexecuted and affordable when a single unit remains, so a root whose
  // Split key bound lies below it can neither reach the cut nor be the last fill.
  if (launch_theta(dm, tv, st, true) != hipSuccess) return GRACEKV_ERR_HIP;
  if (build(BUILD_ROOT_SPLIT) != hipSuccess) return GRACEKV_ERR_HIP;
  if (launch_theta(dm, tv, st, false) != hipSuccess) return GRACEKV_ERR_HIP;
  return hip_status(build(BUILD_CONTINUE));
}

gracekv_status gracekv_score(const gracekv_config* c, const float* omega_raw, void* trees, void* stream) {
  gracekv_plan p;
  gracekv_status s = prep(c, &p);
  if (s != GRACEKV_OK) return s;
  if (!trees || !aligned16(trees)) return GRACEKV_ERR_INVALID_ARG;
  Dims dm = make_dims(*c, p);
  return hip_status(launch_score(dm, omega_raw, make_view(trees, p), (hipStream_t)stream));
}

gracekv_status gracekv_select(const gracekv_config* c, void* trees, int64_t* b_used, void* ws, size_t ws_bytes,
                              void* stream) {
  gracekv_plan p;
  gracekv_status s = prep(c, &p);
  if (s != GRACEKV_OK) return s;
  if (!trees || !b_used || !ws || !aligned16(trees) || !aligned16(ws)) return GRACEKV_ERR_INVALID_ARG;
  if (ws_bytes < p.sel_ws_bytes) return GRACEKV_ERR_WORKSPACE;
  Dims dm = make_dims(*c, p);
  TreeView tv = make_view(trees, p);
  if (c->alpha_floor > 0.0) {                 // the floor's realisation, then the auction from it
    const FloorView fv = floor_of(trees, dm, p, &tv);
    const int clk = clock_begin(dm, GRACEKV_STAGE_FLOOR_REALISE, (hipStream_t)stream);
    const hipError_t e = launch_floor_realise(dm, tv, fv, (hipStream_t)stream);
    clock_end(clk, (hipStream_t)stream);
    if (e != hipSuccess) return GRACEKV_ERR_HIP;
  }
  return hip_status(launch_select(dm, tv, b_used, ws, (hipStream_t)stream));
}

gracekv_status gracekv_pack(const gracekv_config* c, const void* K, const void* V, const float* rope_cos,
                            const float* rope_sin, void* trees, int64_t* offsets, int64_t* counts, void* K_out,
                            void* V_out, int32_t* pos_out, float* logm_out, void* ws, size_t ws_bytes, void* stream) {
  gracekv_plan p;
  gracekv_status s = prep(c, &p);
  if (s != GRACEKV_OK) return s;
  if (!K || !V || !rope_cos || !rope_sin || !trees || !offsets || !counts || !K_out || !V_out || !pos_out ||
      !logm_out || !ws)
    return GRACEKV_ERR_INVALID_ARG;
  if (!aligned16(K) || !aligned16(V) || !aligned16(trees) || !aligned16(ws) || !aligned16(K_out) || !aligned16(V_out))
    return GRACEKV_ERR_INVALID_ARG;
  if (ws_bytes < p.pack_ws_bytes) return GRACEKV_ERR_WORKSPACE;
  Dims dm = make_dims(*c, p);
  return hip_status(launch_pack(dm, K, V, rope_cos, rope_sin, make_view(trees, p), offsets, counts, K_out, V_out,
                                pos_out, logm_out, ws, (hipStream_t)stream));
}

gracekv_status gracekv_relevance_stats(const gracekv_config* c, const void* K, const void* Q, void* trees,
                                       void* stream) {
  gracekv_plan p;
  gracekv_status s = prep(c, &p);
  if (s != GRACEKV_OK) return s;
  if (!K || !Q || !trees || !aligned16(K) || !aligned16(Q) || !aligned16(trees)) return GRACEKV_ERR_INVALID_ARG;
  const Dims dm = make_dims(*c, p);
  const TreeView tv = make_view(trees, p);
  const int clk = clock_begin(dm, GRACEKV_STAGE_ROWSTATS, (hipStream_t)stream);
  const hipError_t e = launch_rowstats(dm, K, Q, tv, (float4*)((char*)trees + p.off_partial), (hipStream_t)stream);
  clock_end(clk, (hipStream_t)stream);
  return hip_status(e);
}

gracekv_status gracekv_decode_ws_bytes(const gracekv_config* c, size_t* ws_bytes) {
  gracekv_plan p;
  gracekv_status s = prep(c, &p);
  if (s != GRACEKV_OK) return s;
  if (!ws_bytes) return GRACEKV_ERR_INVALID_ARG;
  const Dims dm = make_dims(*c, p);
  *ws_bytes = decode_ws_bytes(dm, decode_parts(dm));
  return GRACEKV_OK;
}

gracekv_status gracekv_decode_attention(const gracekv_config* c, const void* q, const int64_t* offsets,
                                        const void* K_out, const void* V_out, const float* logm_out, const void* K,
                                        const void* V, float* out, void* ws, size_t ws_bytes, void* stream) {
  gracekv_plan p;
  gracekv_status s = prep(c, &p);
  if (s != GRACEKV_OK) return s;
  if (!q || !offsets || !K_out || !V_out || !logm_out || !K || !V || !out || !ws) return GRACEKV_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(K_out) || !aligned16(V_out) || !aligned16(K) || !aligned16(V) || !aligned16(ws))
    return GRACEKV_ERR_INVALID_ARG;
  const Dims dm = make_dims(*c, p);
  if (ws_bytes < decode_ws_bytes(dm, decode_parts(dm))) return GRACEKV_ERR_WORKSPACE;
  return hip_status(launch_decode(dm, q, offsets, K_out, V_out, logm_out, K, V, out, ws, (hipStream_t)stream));
}

gracekv_status gracekv_decode_attention_noalloc(const gracekv_config* c, const void* q, const int64_t* offsets,
                                                const void* K_out, const void* V_out, const float* logm_out,
                                                const void* K, const void* V, float* out, void* stream) {
  gracekv_plan p;
  gracekv_status s = prep(c, &p);
  if (s != GRACEKV_OK) return s;
  if (!q || !offsets || !K_out || !V_out || !logm_out || !K || !V || !out) return GRACEKV_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(K_out) || !aligned16(V_out) || !aligned16(K) || !aligned16(V))
    return GRACEKV_ERR_INVALID_ARG;
  const Dims dm = make_dims(*c, p);
  if (decode_ws_bytes(dm, decode_parts(dm)) > (size_t)GRACEKV_DECODE_SCRATCH_BYTES) return GRACEKV_ERR_WORKSPACE;
  return hip_status(launch_decode_noalloc(dm, q, offsets, K_out, V_out, logm_out, K, V, out, (hipStream_t)stream));
}

gracekv_status gracekv_selftest_mfma(int32_t which, float* out, void* stream) {
  if (!out || !aligned16(out) || which < 0 || which > 3) return GRACEKV_ERR_INVALID_ARG;
  return hip_status(selftest_mfma(which, out, (hipStream_t)stream));
}

}  // extern "C"
