// C ABI of libepl: host-side argument checks, layout geometry, workspace sizing and kernel
// launches on the caller's stream. Stateless and reentrant; allocates nothing.
#include <limits.h>

#include <mutex>

#include "epl_internal.h"

#define EPL_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p % a) == 0; }

int bits_for(int n) {  // bits needed to represent values 0..n-1
  int b = 0;
  while ((1 << b) < n) ++b;
  return b;
}

// Common config checks; EPL_OK if the shape is one the library handles.
epl_status check_config(const epl_config* cfg) {
  if (!cfg) return EPL_ERR_INVALID_ARG;
  const int R = cfg->num_ranks, E = cfg->num_experts, k = cfg->topk, H = cfg->hidden, Tr = cfg->tokens_per_rank;
  if (R < 1 || E < R || E > EPL_MAX_EXPERTS || E % R != 0) return EPL_ERR_INVALID_ARG;
  if (k < 1 || k > EPL_MAX_TOPK || Tr < 0 || H < 8 || H > EPL_MAX_HIDDEN || H % 8 != 0) return EPL_ERR_INVALID_ARG;
  if ((int64_t)R * Tr * k >= (int64_t)INT_MAX) return EPL_ERR_INVALID_ARG;
  const int P = cfg->row_pitch;
  if (P != 0 && (P < H || P > EPL_MAX_HIDDEN || P % 64 != 0)) return EPL_ERR_INVALID_ARG;
  if (cfg->payload != EPL_PAYLOAD_BF16 && cfg->payload != EPL_PAYLOAD_FP8_E4M3) return EPL_ERR_UNSUPPORTED;
  return EPL_OK;
}

// Elements from one receive (and expert-output) row to the next.
int pitch_of(const epl_config* cfg) { return cfg->row_pitch ? cfg->row_pitch : cfg->hidden; }

// Chunking of each source rank's tokens for the layout kernels: whole tokens, at most
// kMaxChunkPairs pairs per workgroup.
epl::Geom make_geom(const epl_config* cfg) {
  epl::Geom g;
  g.R = cfg->num_ranks;
  g.E = cfg->num_experts;
  g.El = g.E / g.R;
  g.k = cfg->topk;
  g.Tr = cfg->tokens_per_rank;
  g.T = (int64_t)g.R * g.Tr;
  // Aim for >= 256 workgroups (the chip has 256 CUs) and >= 64 pairs per workgroup, with at
  // most kMaxChunkPairs pairs per chunk.
  const int cap = epl::kMaxChunkPairs / g.k;  // k <= 32 so cap >= 32
  const int64_t want = std::max<int64_t>((g.T + 255) / 256, (64 + g.k - 1) / g.k);
  const int ct = (int)std::min<int64_t>(want, cap);
  g.CT = g.Tr < 1 ? 1 : std::min(ct, g.Tr);
  g.NC = g.Tr < 1 ? 1 : (g.Tr + g.CT - 1) / g.CT;
  g.nblk = g.R * g.NC;
  g.ebits = bits_for(g.E);
  g.rbits = bits_for(g.R);
  g.inv_k = 1.0f / (float)g.k;
  g.inv_El = 1.0f / (float)g.El;
  g.inv_R = 1.0f / (float)g.R;
  return g;
}

size_t workspace_bytes(const epl::Geom& g) { return epl::ws_layout(g).total * sizeof(int32_t); }

epl_status check_layout_buffers(const epl_layout_buffers* L) {
  if (!L) return EPL_ERR_INVALID_ARG;
  int32_t* const ptrs[] = {L->send_cnt, L->rank_cnt, L->expert_off, L->rank_off, L->seg_off, L->tok_nranks,
                           L->pair_row, L->pair_rslot, L->recv_src,  L->recv_j,   L->num_invalid};
  for (int32_t* p : ptrs) {
    if (!p) return EPL_ERR_INVALID_ARG;
    if (!aligned(p, 4)) return EPL_ERR_ALIGN;
  }
  return EPL_OK;
}

epl_status from_hip(hipError_t e) { return e == hipSuccess ? EPL_OK : EPL_ERR_DEVICE; }

}  // namespace

EPL_EXPORT size_t epl_workspace_bytes(const epl_config* cfg) {
  if (check_config(cfg) != EPL_OK) return 0;
  return workspace_bytes(make_geom(cfg));
}

namespace {

// The checks of epl_layout (topk_idx, L, workspace), shared by the calls that run the layout.
epl_status check_layout_args(const epl_config* cfg, const int32_t* topk_idx, const epl_layout_buffers* L,
                             void* workspace, size_t ws_bytes) {
  epl_status st = check_config(cfg);
  if (st != EPL_OK) return st;
  if ((st = check_layout_buffers(L)) != EPL_OK) return st;
  const epl::Geom g = make_geom(cfg);
  if (g.T > 0 && !topk_idx) return EPL_ERR_INVALID_ARG;
  if (!aligned(topk_idx, 4)) return EPL_ERR_ALIGN;
  if (!workspace) return EPL_ERR_WORKSPACE;
  if (!aligned(workspace, 4)) return EPL_ERR_ALIGN;
  if (ws_bytes < workspace_bytes(g)) return EPL_ERR_WORKSPACE;
  return EPL_OK;
}

// The layout checks plus those of epl_dispatch (x, recv, recv_scale, capacity).
epl_status check_layout_dispatch(const epl_config* cfg, const int32_t* topk_idx, const epl_layout_buffers* L,
                                 void* workspace, size_t ws_bytes, const void* x, void* recv, float* recv_scale,
                                 int64_t recv_rows_cap) {
  epl_status st = check_config(cfg);
  if (st != EPL_OK) return st;
  const bool fp8 = cfg->payload == EPL_PAYLOAD_FP8_E4M3;
  if (fp8 && cfg->hidden % 128 != 0) return EPL_ERR_UNSUPPORTED;
  if ((st = check_layout_args(cfg, topk_idx, L, workspace, ws_bytes)) != EPL_OK) return st;
  const epl::Geom g = make_geom(cfg);
  if (g.T > 0 && (!x || !recv || (fp8 && !recv_scale))) return EPL_ERR_INVALID_ARG;
  if (!aligned(x, 16) || !aligned(recv, 16) || (fp8 && !aligned(recv_scale, 4))) return EPL_ERR_ALIGN;
  if (recv_rows_cap < g.T * cfg->topk) return EPL_ERR_CAPACITY;
  return EPL_OK;
}

bool rows_fused(const epl::Geom& g, const epl_config* cfg) {
  return !epl::layout_single(g) && epl::fused_dispatch_ok(g, cfg->payload == EPL_PAYLOAD_FP8_E4M3);
}

// The layout kernels the row kernel does not take over: histogram and scan when the finalize
// step is fused into the row kernel, otherwise the whole layout.
hipError_t run_counts(const epl::Geom& g, const epl_config* cfg, const int32_t* topk_idx,
                      const epl_layout_buffers* L, int32_t* ws, hipStream_t s) {
  if (rows_fused(g, cfg))
    return epl::launch_layout_counts(g, topk_idx, ws, L->send_cnt, L->rank_cnt, L->tok_nranks, L->num_invalid, s);
  return epl::launch_layout(g, topk_idx, ws, L->send_cnt, L->rank_cnt, L->expert_off, L->rank_off, L->seg_off,
                            L->tok_nranks, L->pair_row, L->pair_rslot, L->recv_src, L->recv_j, L->num_invalid, s);
}

// One kernel: the fused finalize-and-send kernel, or the plain bf16 / fp8 dispatch kernel.
hipError_t run_rows(const epl::Geom& g, const epl_config* cfg, const int32_t* topk_idx, const epl_layout_buffers* L,
                    int32_t* ws, const void* x, void* recv, float* recv_scale, int64_t cap, hipStream_t s) {
  if (rows_fused(g, cfg))
    return epl::launch_fused_dispatch(g, topk_idx, ws, L->expert_off, L->rank_off, L->seg_off, L->pair_row,
                                      L->pair_rslot, L->recv_src, L->recv_j, x, recv, cfg->hidden, pitch_of(cfg),
                                      cap, s);
  if (cfg->payload == EPL_PAYLOAD_FP8_E4M3)
    return epl::launch_dispatch_fp8(x, L->pair_row, recv, recv_scale, g.T, cfg->topk, cfg->hidden, pitch_of(cfg),
                                    cap, s);
  return epl::launch_dispatch_bf16(x, L->pair_row, recv, g.T, cfg->topk, cfg->hidden, pitch_of(cfg), cap, s);
}

}  // namespace

EPL_EXPORT epl_status epl_layout(const epl_config* cfg, const int32_t* topk_idx, const epl_layout_buffers* L,
                                 void* workspace, size_t ws_bytes, void* stream) {
  const epl_status st = check_layout_args(cfg, topk_idx, L, workspace, ws_bytes);
  if (st != EPL_OK) return st;
  return from_hip(epl::launch_layout(make_geom(cfg), topk_idx, static_cast<int32_t*>(workspace), L->send_cnt,
                                     L->rank_cnt, L->expert_off, L->rank_off, L->seg_off, L->tok_nranks, L->pair_row,
                                     L->pair_rslot, L->recv_src, L->recv_j, L->num_invalid,
                                     static_cast<hipStream_t>(stream)));
}

EPL_EXPORT epl_status epl_dispatch(const epl_config* cfg, const void* x, const epl_layout_buffers* L, void* recv,
                                   float* recv_scale, int64_t recv_rows_cap, void* stream) {
  epl_status st = check_config(cfg);
  if (st != EPL_OK) return st;
  const bool fp8 = cfg->payload == EPL_PAYLOAD_FP8_E4M3;
  if (fp8 && cfg->hidden % 128 != 0) return EPL_ERR_UNSUPPORTED;
  if (!L || !L->pair_row) return EPL_ERR_INVALID_ARG;
  if (!aligned(L->pair_row, 4)) return EPL_ERR_ALIGN;
  const int64_t T = (int64_t)cfg->num_ranks * cfg->tokens_per_rank;
  if (T > 0 && (!x || !recv || (fp8 && !recv_scale))) return EPL_ERR_INVALID_ARG;
  if (!aligned(x, 16) || !aligned(recv, 16) || (fp8 && !aligned(recv_scale, 4))) return EPL_ERR_ALIGN;
  if (recv_rows_cap < T * cfg->topk) return EPL_ERR_CAPACITY;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (fp8) return from_hip(epl::launch_dispatch_fp8(x, L->pair_row, recv, recv_scale, T, cfg->topk, cfg->hidden,
                                                   pitch_of(cfg), recv_rows_cap, s));
  return from_hip(epl::launch_dispatch_bf16(x, L->pair_row, recv, T, cfg->topk, cfg->hidden, pitch_of(cfg),
                                            recv_rows_cap, s));
}


EPL_EXPORT epl_status epl_layout_counts(const epl_config* cfg, const int32_t* topk_idx, const epl_layout_buffers* L,
                                        void* workspace, size_t ws_bytes, void* stream) {
  const epl_status st = check_layout_args(cfg, topk_idx, L, workspace, ws_bytes);
  if (st != EPL_OK) return st;
  return from_hip(run_counts(make_geom(cfg), cfg, topk_idx, L, static_cast<int32_t*>(workspace),
                             static_cast<hipStream_t>(stream)));
}

EPL_EXPORT epl_status epl_dispatch_rows(const epl_config* cfg, const int32_t* topk_idx, const epl_layout_buffers* L,
                                        void* workspace, size_t ws_bytes, const void* x, void* recv,
                                        float* recv_scale, int64_t recv_rows_cap, void* stream) {
  const epl_status st =
      check_layout_dispatch(cfg, topk_idx, L, workspace, ws_bytes, x, recv, recv_scale, recv_rows_cap);
  if (st != EPL_OK) return st;
  return from_hip(run_rows(make_geom(cfg), cfg, topk_idx, L, static_cast<int32_t*>(workspace), x, recv, recv_scale,
                           recv_rows_cap, static_cast<hipStream_t>(stream)));
}

EPL_EXPORT epl_status epl_layout_dispatch(const epl_config* cfg, const int32_t* topk_idx, const epl_layout_buffers* L,
                                          void* workspace, size_t ws_bytes, const void* x, void* recv,
                                          float* recv_scale, int64_t recv_rows_cap, void* stream) {
  const epl_status st =
      check_layout_dispatch(cfg, topk_idx, L, workspace, ws_bytes, x, recv, recv_scale, recv_rows_cap);
  if (st != EPL_OK) return st;
  const epl::Geom g = make_geom(cfg);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t* ws = static_cast<int32_t*>(workspace);
  const hipError_t e = run_counts(g, cfg, topk_idx, L, ws, s);
  if (e != hipSuccess) return from_hip(e);
  return from_hip(run_rows(g, cfg, topk_idx, L, ws, x, recv, recv_scale, recv_rows_cap, s));
}

// ------------------------------------------------------------------ decomposed single launch
namespace {

epl_status decomposed_args(const epl_config* cfg, const epl_decomposed_opts* opts, epl::DecomposedOpts* out) {
  epl::DecomposedOpts o{0, 0, 1};
  int64_t spin_us = 100000;
  if (opts) {
    if (opts->count_groups < 0 || opts->spin_limit_us < 0 || opts->test_ready_target < 0) return EPL_ERR_INVALID_ARG;
    o.count_groups = opts->count_groups;
    if (opts->spin_limit_us > 0) spin_us = opts->spin_limit_us;
    if (opts->test_ready_target > 0) o.ready_target = opts->test_ready_target;
  }
  o.spin_ticks = spin_us * 100;  // the real-time clock runs at 100 MHz
  if (cfg->payload != EPL_PAYLOAD_BF16 || !epl::fused_dispatch_ok(make_geom(cfg), false)) return EPL_ERR_UNSUPPORTED;
  *out = o;
  return EPL_OK;
}

}  // namespace

EPL_EXPORT epl_status epl_layout_dispatch_decomposed(const epl_config* cfg, const int32_t* topk_idx,
                                                     const epl_layout_buffers* L, void* workspace, size_t ws_bytes,
                                                     const void* x, void* recv, float* recv_scale,
                                                     int64_t recv_rows_cap, const epl_decomposed_opts* opts,
                                                     int32_t* wait_status, void* stream) {
  epl_status st = check_layout_dispatch(cfg, topk_idx, L, workspace, ws_bytes, x, recv, recv_scale, recv_rows_cap);
  if (st != EPL_OK) return st;
  epl::DecomposedOpts o;
  if ((st = decomposed_args(cfg, opts, &o)) != EPL_OK) return st;
  if (!wait_status) return EPL_ERR_INVALID_ARG;
  if (!aligned(wait_status, 4)) return EPL_ERR_ALIGN;
  const epl::Geom g = make_geom(cfg);
  epl::DecomposedPlan plan;
  if (epl::plan_decomposed(g, cfg->hidden, o.count_groups, epl::kDafNone, &plan) != hipSuccess) return EPL_ERR_DEVICE;
  if (plan.grid > plan.capacity) return EPL_ERR_UNSUPPORTED;
  return from_hip(epl::launch_decomposed(g, topk_idx, static_cast<int32_t*>(workspace), *L, x, recv, cfg->hidden,
                                         pitch_of(cfg), recv_rows_cap, o, wait_status,
                                         static_cast<hipStream_t>(stream)));
}

EPL_EXPORT int epl_decomposed_plan(const epl_config* cfg, int32_t count_groups, int32_t* grid, int32_t* capacity) {
  if (check_config(cfg) != EPL_OK || count_groups < 0) return -1;
  if (cfg->payload != EPL_PAYLOAD_BF16 || !epl::fused_dispatch_ok(make_geom(cfg), false)) return -1;
  epl::DecomposedPlan plan;
  if (epl::plan_decomposed(make_geom(cfg), cfg->hidden, count_groups, epl::kDafNone, &plan) != hipSuccess) return -1;
  if (grid) *grid = plan.grid;
  if (capacity) *capacity = plan.capacity;
  return plan.count_groups;
}

namespace {

// The checks and the launch shared by the one-launch layer calls (Sentinel Polling, and the
// flag and checksum variants).
epl_status run_layer(const epl_config* cfg, const int32_t* topk_idx, const epl_layout_buffers* L, void* workspace,
                     size_t ws_bytes, const void* x, void* recv, int64_t recv_rows_cap, const float* topk_w, void* out,
                     const epl_decomposed_opts* opts, int32_t* wait_status, void* stream, int sync, uint64_t* marks,
                     uint64_t epoch) {
  epl_status st = check_layout_dispatch(cfg, topk_idx, L, workspace, ws_bytes, x, recv, nullptr, recv_rows_cap);
  if (st != EPL_OK) return st;
  epl::DecomposedOpts o;
  if ((st = decomposed_args(cfg, opts, &o)) != EPL_OK) return st;
  const epl::Geom g = make_geom(cfg);
  if (g.T > 0 && (!topk_w || !out)) return EPL_ERR_INVALID_ARG;
  if (!wait_status) return EPL_ERR_INVALID_ARG;
  if (!aligned(wait_status, 4) || !aligned(topk_w, 4) || !aligned(out, 16)) return EPL_ERR_ALIGN;
  if (sync != epl::kDafSentinel) {
    if (g.T > 0 && !marks) return EPL_ERR_INVALID_ARG;
    if (!aligned(marks, 8)) return EPL_ERR_ALIGN;
    if (epoch == 0) return EPL_ERR_INVALID_ARG;
  }
  epl::DecomposedPlan plan;
  if (epl::plan_decomposed(g, cfg->hidden, o.count_groups, sync, &plan) != hipSuccess) return EPL_ERR_DEVICE;
  if (plan.grid > plan.capacity) return EPL_ERR_UNSUPPORTED;
  return from_hip(epl::launch_decomposed(g, topk_idx, static_cast<int32_t*>(workspace), *L, x, recv, cfg->hidden,
                                         pitch_of(cfg), recv_rows_cap, o, wait_status,
                                         static_cast<hipStream_t>(stream), sync, topk_w, out, marks, epoch));
}

}  // namespace

EPL_EXPORT epl_status epl_layer_sentinel(const epl_config* cfg, const int32_t* topk_idx, const epl_layout_buffers* L,
                                         void* workspace, size_t ws_bytes, const void* x, void* recv,
                                         int64_t recv_rows_cap, const float* topk_w, void* out,
                                         const epl_decomposed_opts* opts, int32_t* wait_status, void* stream) {
  return run_layer(cfg, topk_idx, L, workspace, ws_bytes, x, recv, recv_rows_cap, topk_w, out, opts, wait_status,
                   stream, epl::kDafSentinel, nullptr, 0);
}

EPL_EXPORT int64_t epl_layer_marks_bytes(const epl_config* cfg, int64_t recv_rows_cap) {
  if (check_config(cfg) != EPL_OK || recv_rows_cap < 0) return -1;
  const int64_t cchunks = (cfg->hidden / 8 + 63) / 64;
  return recv_rows_cap * cchunks * (int64_t)sizeof(uint64_t);
}

EPL_EXPORT epl_status epl_layer_data_as_flag(const epl_config* cfg, const int32_t* topk_idx,
                                             const epl_layout_buffers* L, void* workspace, size_t ws_bytes,
                                             const void* x, void* recv, int64_t recv_rows_cap, const float* topk_w,
                                             void* out, uint64_t* marks, int32_t variant, uint64_t epoch,
                                             const epl_decomposed_opts* opts, int32_t* wait_status, void* stream) {
  int sync;
  if (variant == EPL_DAF_TOKEN_FLAG_FUSION)
    sync = epl::kDafFlag;
  else if (variant == EPL_DAF_DATA_CHECKSUM)
    sync = epl::kDafChecksum;
  else
    return check_config(cfg) != EPL_OK ? check_config(cfg) : EPL_ERR_INVALID_ARG;
  return run_layer(cfg, topk_idx, L, workspace, ws_bytes, x, recv, recv_rows_cap, topk_w, out, opts, wait_status,
                   stream, sync, marks, epoch);
}

EPL_EXPORT epl_status epl_sentinel_fill(void* buf, int64_t n, void* stream) {
  if (n < 0 || n % 8 != 0 || (n > 0 && !buf)) return EPL_ERR_INVALID_ARG;
  if (!aligned(buf, 16)) return EPL_ERR_ALIGN;
  return from_hip(epl::launch_sentinel_fill(buf, n / 8, static_cast<hipStream_t>(stream)));
}

EPL_EXPORT int64_t epl_sentinel_find(const uint16_t* values, int64_t n) {
  if (!values || n <= 0) return -1;
  for (int64_t i = 0; i < n; ++i)
    if (values[i] == EPL_SENTINEL_BF16) return i;
  return -1;
}

// ------------------------------------------------------------------ allocation-free variant
// The layout workspace of epl_layout_dispatch_noalloc: one array per GPU, held by the loaded
// library until the process ends. In host code `scratch` names a host-side stand-in, never the
// device address; that comes from hipGetSymbolAddress, taken once per device with the device
// current and kept in g_scratch.
static __device__ __align__(256) int32_t scratch[EPL_STATIC_SCRATCH_BYTES / sizeof(int32_t)];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
int32_t* g_scratch[kMaxDevices] = {};

// The device address of this GPU's scratch array (looked up on the first call for the device).
hipError_t device_scratch(hipStream_t stream, int32_t** out) {
  int dev = 0;
  hipError_t e = stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    int cur = 0;
    if ((e = hipGetDevice(&cur)) != hipSuccess) return e;
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) {
      const hipError_t e2 = hipSetDevice(cur);
      if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch[dev] = static_cast<int32_t*>(p);
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

}  // namespace

EPL_EXPORT epl_status epl_layout_dispatch_noalloc(const epl_config* cfg, const int32_t* topk_idx,
                                                  const epl_layout_buffers* L, const void* x, void* recv,
                                                  float* recv_scale, int64_t recv_rows_cap, void* stream) {
  epl_status st = check_config(cfg);
  if (st != EPL_OK) return st;
  const epl::Geom g = make_geom(cfg);
  if (workspace_bytes(g) > (size_t)EPL_STATIC_SCRATCH_BYTES) return EPL_ERR_WORKSPACE;
  // The other checks are those of epl_layout_dispatch, with the static array as the workspace
  // (a 256-byte aligned stand-in pointer passes the workspace checks; it is never dereferenced).
  st = check_layout_dispatch(cfg, topk_idx, L, reinterpret_cast<void*>(256), (size_t)EPL_STATIC_SCRATCH_BYTES, x,
                             recv, recv_scale, recv_rows_cap);
  if (st != EPL_OK) return st;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t* ws = nullptr;
  hipError_t e = device_scratch(s, &ws);
  if (e != hipSuccess) return from_hip(e);
  e = run_counts(g, cfg, topk_idx, L, ws, s);
  if (e != hipSuccess) return from_hip(e);
  return from_hip(run_rows(g, cfg, topk_idx, L, ws, x, recv, recv_scale, recv_rows_cap, s));
}

EPL_EXPORT int epl_layout_dispatch_launches(const epl_config* cfg) {
  if (check_config(cfg) != EPL_OK) return -1;
  const epl::Geom g = make_geom(cfg);
  if (epl::layout_single(g)) return 2;
  return epl::fused_dispatch_ok(g, cfg->payload == EPL_PAYLOAD_FP8_E4M3) ? 3 : 4;
}

EPL_EXPORT epl_status epl_locate_rows(const epl_config* cfg, const int32_t* expert_off, const int32_t* rows,
                                      int64_t n, int32_t* expert, int32_t* offset, void* stream) {
  const epl_status st = check_config(cfg);
  if (st != EPL_OK) return st;
  if (n < 0) return EPL_ERR_INVALID_ARG;
  if (n > 0 && (!expert_off || !expert || !offset)) return EPL_ERR_INVALID_ARG;
  if (!aligned(expert_off, 4) || !aligned(rows, 4) || !aligned(expert, 4) || !aligned(offset, 4)) return EPL_ERR_ALIGN;
  return from_hip(epl::launch_locate_rows(expert_off, rows, n, cfg->num_experts, expert, offset,
                                          static_cast<hipStream_t>(stream)));
}

EPL_EXPORT epl_status epl_hop_schedule(const epl_config* cfg, const int32_t* send_cnt, const int32_t* order,
                                       int32_t remap_rows, const int32_t* hop_class, int32_t workers,
                                       int32_t num_classes, int32_t* start_expert, int32_t* start_offset,
                                       int32_t* class_cnt, void* stream) {
  const epl_status st = check_config(cfg);
  if (st != EPL_OK) return st;
  if (workers < 1 || (int64_t)cfg->num_ranks * workers >= (int64_t)INT_MAX || remap_rows < 0 || num_classes < 1 ||
      num_classes > EPL_MAX_HOP_CLASSES)
    return EPL_ERR_INVALID_ARG;
  if (!send_cnt || !hop_class || !start_expert || !start_offset || !class_cnt) return EPL_ERR_INVALID_ARG;
  const void* ptrs[] = {send_cnt, order, hop_class, start_expert, start_offset, class_cnt};
  for (const void* p : ptrs)
    if (!aligned(p, 4)) return EPL_ERR_ALIGN;
  return from_hip(epl::launch_hop_schedule(send_cnt, order, hop_class, cfg->num_ranks, cfg->num_experts,
                                           remap_rows ? remap_rows : workers, workers, num_classes, start_expert,
                                           start_offset, class_cnt, static_cast<hipStream_t>(stream)));
}

EPL_EXPORT epl_status epl_dispatch_scheduled(const epl_config* cfg, const void* x, const epl_layout_buffers* L,
                                             void* recv, float* recv_scale, int64_t recv_rows_cap, int32_t remap_rows,
                                             int32_t workers, void* stream) {
  const epl_status st = check_config(cfg);
  if (st != EPL_OK) return st;
  const bool fp8 = cfg->payload == EPL_PAYLOAD_FP8_E4M3;
  if (fp8 && cfg->hidden % 128 != 0) return EPL_ERR_UNSUPPORTED;
  if (workers < 1 || (int64_t)cfg->num_ranks * workers >= (int64_t)INT_MAX || remap_rows < 0)
    return EPL_ERR_INVALID_ARG;
  if (!L || !L->send_cnt || !L->seg_off || !L->recv_src) return EPL_ERR_INVALID_ARG;
  if (!aligned(L->send_cnt, 4) || !aligned(L->seg_off, 4) || !aligned(L->recv_src, 4)) return EPL_ERR_ALIGN;
  const int64_t T = (int64_t)cfg->num_ranks * cfg->tokens_per_rank;
  if (T > 0 && (!x || !recv || (fp8 && !recv_scale))) return EPL_ERR_INVALID_ARG;
  if (!aligned(x, 16) || !aligned(recv, 16) || (fp8 && !aligned(recv_scale, 4))) return EPL_ERR_ALIGN;
  if (recv_rows_cap < T * cfg->topk) return EPL_ERR_CAPACITY;
  return from_hip(epl::launch_dispatch_scheduled(x, L->send_cnt, L->seg_off, L->recv_src, recv,
                                                 fp8 ? recv_scale : nullptr, cfg->num_ranks, cfg->num_experts,
                                                 remap_rows ? remap_rows : workers, workers, T, cfg->topk,
                                                 cfg->hidden, pitch_of(cfg), recv_rows_cap,
                                                 static_cast<hipStream_t>(stream)));
}

EPL_EXPORT epl_status epl_combine(const epl_config* cfg, const void* y, const float* topk_w,
                                  const epl_layout_buffers* L, void* out, void* stream) {
  epl_status st = check_config(cfg);
  if (st != EPL_OK) return st;
  if (!L || !L->pair_row) return EPL_ERR_INVALID_ARG;
  if (!aligned(L->pair_row, 4)) return EPL_ERR_ALIGN;
  const int64_t T = (int64_t)cfg->num_ranks * cfg->tokens_per_rank;
  if (T > 0 && (!y || !topk_w || !out)) return EPL_ERR_INVALID_ARG;
  if (!aligned(y, 16) || !aligned(out, 16) || !aligned(topk_w, 4)) return EPL_ERR_ALIGN;
  return from_hip(epl::launch_combine(y, topk_w, L->pair_row, out, T, cfg->topk, cfg->hidden, pitch_of(cfg),
                                      static_cast<hipStream_t>(stream)));
}

EPL_EXPORT epl_status epl_debug_f32_to_e4m3(const float* in, uint8_t* out, int64_t n, void* stream) {
  if (n < 0 || (n > 0 && (!in || !out))) return EPL_ERR_INVALID_ARG;
  if (!aligned(in, 4) || !aligned(out, 4)) return EPL_ERR_ALIGN;
  return from_hip(epl::launch_debug_e4m3(in, out, n, static_cast<hipStream_t>(stream)));
}

EPL_EXPORT epl_status epl_debug_f32_to_bf16(const float* in, uint16_t* out, int64_t n, void* stream) {
  if (n < 0 || (n > 0 && (!in || !out))) return EPL_ERR_INVALID_ARG;
  if (!aligned(in, 4) || !aligned(out, 4)) return EPL_ERR_ALIGN;
  return from_hip(epl::launch_debug_bf16(in, out, n, static_cast<hipStream_t>(stream)));
}

EPL_EXPORT const char* epl_status_str(epl_status s) {
  switch (s) {
    case EPL_OK: return "EPL_OK";
    case EPL_ERR_INVALID_ARG: return "EPL_ERR_INVALID_ARG: invalid argument";
    case EPL_ERR_ALIGN: return "EPL_ERR_ALIGN: misaligned pointer";
    case EPL_ERR_CAPACITY: return "EPL_ERR_CAPACITY: recv_rows_cap < T*k";
    case EPL_ERR_WORKSPACE: return "EPL_ERR_WORKSPACE: workspace too small";
    case EPL_ERR_UNSUPPORTED: return "EPL_ERR_UNSUPPORTED: unsupported payload or hidden size";
    case EPL_ERR_DEVICE: return "EPL_ERR_DEVICE: HIP runtime error";
  }
  return "EPL: unknown status";
}

EPL_EXPORT int epl_layout_launches(const epl_config* cfg) {
  if (check_config(cfg) != EPL_OK) return -1;
  return epl::layout_single(make_geom(cfg)) ? 1 : 3;
}

EPL_EXPORT const char* epl_version(void) { return "epl 0.1.0 (gfx950)"; }
