// Internal declarations shared by the epl HIP sources (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <stddef.h>
#include <stdint.h>

#include "epl.h"

namespace epl {

constexpr int kWave = 64;
constexpr int kLayoutThreads = 256;
constexpr int kLayoutWaves = kLayoutThreads / kWave;
// Pairs handled by one layout workgroup ("chunk"); a chunk never spans two source ranks and
// always holds whole tokens.
constexpr int kMaxChunkPairs = 1024;
constexpr int kChunkSlots = kMaxChunkPairs / kLayoutThreads;  // register slots per lane
constexpr int kLayoutSlots = EPL_MAX_EXPERTS / kLayoutThreads;  // per-lane slots covering E or R experts/ranks
// The single-launch layout reads all T*k ids in every workgroup and walks each source rank's
// earlier tokens again, so it is used only up to these sizes; larger layouts take three launches.
// Measured on MI355X, the one-launch layout costs about 11 us + 12 us per 64K pairs, against
// 17-22 us for three launches: it wins up to about 37K pairs.
constexpr int64_t kSingleMaxPairs = 16384;     // T*k
constexpr int64_t kSingleMaxRankPairs = 4096;  // Tr*k
constexpr size_t kSingleMaxLds = 64 * 1024;    // bytes of LDS per workgroup

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Buffer resource descriptor word 3 for raw (untyped) buffer accesses on CDNA3/CDNA4.
constexpr int kBufferRsrcWord3 = 0x00020000;
// Cache-policy operand of the raw buffer builtins: bit 0 = sc0, bit 1 = nt, bit 4 = sc1.
constexpr int kCachePolicySc1 = 16;
constexpr int kCachePolicySc1Nt = 18;

// Shape of one layout problem, derived on the host from epl_config.
struct Geom {
  int R, E, El, k, Tr;
  int CT;     // tokens per chunk
  int NC;     // chunks per source rank (>= 1)
  int nblk;   // R * NC layout workgroups
  int ebits;  // bits needed for an expert id (ballot-match key width)
  int rbits;  // bits needed for a rank id
  float inv_k, inv_El, inv_R;  // 1/k, 1/El, 1/R for exact small quotients
  int64_t T;
};

// Workspace carve-up, in int32 elements.
struct WsLayout {
  size_t chunk_e;   // [E][nblk]  per-chunk expert counts, then chunk base rows within the expert
  size_t chunk_r;   // [nblk][R]  per-chunk first-pair counts per destination rank, then slot bases
  size_t recv_cnt;  // [E]
  size_t inval;     // [nblk]
  size_t seg_rel;   // [E][R]     segment offsets relative to the expert start
  size_t fmask;     // [T]        per-token bitmask of first pairs per destination rank
  size_t cnt;       // [nblk][E]  per-chunk expert counts, chunk-major (the decomposed layer's K1 rows)
  size_t sync;      // [kSyncWords] completion words of the decomposed layer, 256-byte aligned
  size_t total;
};
// Words of the decomposed single-launch layer's synchronisation: zero before its first call on a
// workspace (a zero-filled workspace), and left zero by every call. Each word the kernel polls or
// counts on sits in a 128-byte line of its own (kSyncStride words apart): one shared line made
// every count and poll contend.
constexpr int kSyncStride = 32;
constexpr int kSyncWords = 8 * kSyncStride;

inline WsLayout ws_layout(const Geom& g) {
  WsLayout w;
  size_t o = 0;
  w.chunk_e = o;
  o += (size_t)g.E * g.nblk;
  w.chunk_r = o;
  o += (size_t)g.nblk * g.R;
  w.recv_cnt = o;
  o += (size_t)g.E;
  w.inval = o;
  o += (size_t)g.nblk;
  w.seg_rel = o;
  o += (size_t)g.E * g.R;
  w.fmask = o;
  o += (size_t)g.T;
  w.cnt = o;
  o += (size_t)g.nblk * g.E;
  o = (o + 63) & ~(size_t)63;
  w.sync = o;
  o += kSyncWords;
  w.total = o;
  return w;
}

// Small integer quotient q = n / d for 0 <= n < 2^21 and the float reciprocal inv_d = 1/d:
// q = (int)((n + 0.5f) * inv_d). The exact quotient sits at least 0.5/d away from an integer, and
// two float roundings perturb (n + 0.5)/d by at most (n + 0.5) * 2^-22 / d, which is smaller than
// 0.5/d. So the truncated result is exact.
__device__ __forceinline__ int small_div(int n, float inv_d) { return (int)(((float)n + 0.5f) * inv_d); }

// ---------------------------------------------------------------- wave64 primitives
__device__ __forceinline__ int lane_id() { return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0)); }

// popcount(mask & lanes-below-me): a lane's rank among the lanes of `mask`.
__device__ __forceinline__ int rank_in_mask(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
}

// Lanes of the wave that are active and hold the same `key` as this lane (match-any built
// from one ballot per key bit). `nbits` must be wave-uniform. Result is meaningless for an
// inactive lane.
__device__ __forceinline__ uint64_t match_key(bool active, int key, int nbits) {
  uint64_t m = __ballot(active);
  for (int b = 0; b < nbits; ++b) {
    const bool bit = (key >> b) & 1;
    const uint64_t bb = __ballot(active && bit);
    m &= bit ? bb : ~bb;
  }
  return m;
}

__device__ __forceinline__ int wave_inclusive_sum(int v) {
  const int lane = lane_id();
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int t = __shfl_up(v, off, kWave);
    if (lane >= off) v += t;
  }
  return v;
}

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

// Exclusive prefix sum across a 256-thread block; `total` receives the block sum. Every
// thread of the block must call it (it synchronises).
__device__ __forceinline__ int block_exclusive_sum(int v, int& total, int* scratch /* [kLayoutWaves] */) {
  const int inc = wave_inclusive_sum(v);
  const int w = threadIdx.x / kWave;
  if (lane_id() == kWave - 1) scratch[w] = inc;
  __syncthreads();
  int pre = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < kLayoutWaves; ++i) {
    const int s = scratch[i];
    pre += (i < w) ? s : 0;
    tot += s;
  }
  __syncthreads();
  total = tot;
  return pre + inc - v;
}

// ---------------------------------------------------------------- quaternary search
// Position lookup over a non-decreasing list of cumulative counts off[0..n] with off[0] = 0
// (Algorithm 1, Quaternary Search, with the loop ending once the window holds one entry): for
// 0 <= t < off[n], the index i with off[i] <= t < off[i + 1], i.e. the non-empty entry whose
// cumulative range covers t. The window [L, R) keeps off[L] <= t < off[R]; a step reads the counts
// at three cut points as independent loads and keeps the quarter that holds t, so it ends after
// ceil(log4 n) steps. off may live in LDS or global memory.
__device__ __forceinline__ int quaternary_find(const int32_t* off, int n, int64_t t) {
  int L = 0, R = n;
  while (R - L > 1) {
    const int gap = (R - L + 3) >> 2;
    const int p1 = min(L + gap, R), p2 = min(L + 2 * gap, R), p3 = min(L + 3 * gap, R);
    const int c1 = off[p1], c2 = off[p2], c3 = off[p3];
    if (t < c1) {
      R = p1;
    } else if (t < c2) {
      L = p1;
      R = p2;
    } else if (t < c3) {
      L = p2;
      R = p3;
    } else {
      L = p3;
    }
  }
  return L;
}

// ---------------------------------------------------------------- number conversions
// Clamp to [-448, 448], letting NaN through: the median of three returns -448 for a NaN.
__device__ __forceinline__ float clamp_e4m3(float v) {
  return __builtin_isnan(v) ? v : __builtin_amdgcn_fmed3f(v, 448.0f, -448.0f);
}

// Bit 7 of byte i set where the i-th value is a NaN with its sign bit clear (as an int32, a
// positive NaN is above the bits of +Inf).
__device__ __forceinline__ uint32_t positive_nan_bytes(float a, float b, float c, float d) {
  uint32_t m = __float_as_int(a) > 0x7F800000 ? 0x00000080u : 0u;
  m |= __float_as_int(b) > 0x7F800000 ? 0x00008000u : 0u;
  m |= __float_as_int(c) > 0x7F800000 ? 0x00800000u : 0u;
  m |= __float_as_int(d) > 0x7F800000 ? 0x80000000u : 0u;
  return m;
}

// Four fp32 values -> four OCP E4M3 bytes (byte i from argument i), round to nearest even,
// magnitudes above 448 saturated to 448 (the clamp is exact and RNE never rounds a value
// below 464 past 448), sign kept on zero, NaN -> 0x7F with its sign. The conversion instruction
// writes 0xFF for every NaN, so the sign bit of a positive NaN's byte is cleared afterwards.
__device__ __forceinline__ uint32_t f32x4_to_e4m3x4(float a, float b, float c, float d) {
  const uint32_t pos_nan = positive_nan_bytes(a, b, c, d);
  a = clamp_e4m3(a);
  b = clamp_e4m3(b);
  c = clamp_e4m3(c);
  d = clamp_e4m3(d);
  const uint32_t lo = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0u, false);
  return __builtin_amdgcn_cvt_pk_fp8_f32(c, d, lo, true) & ~pos_nan;
}

// Two fp32 -> packed bf16x2 (low half from `lo`), round to nearest even.
__device__ __forceinline__ uint32_t f32x2_to_bf16x2(float lo, float hi) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const f32x2 f = {lo, hi};
  const bf16x2 b = __builtin_convertvector(f, bf16x2);
  return __builtin_bit_cast(uint32_t, b);
}

__device__ __forceinline__ float bf16lo_to_f32(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi_to_f32(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// ---------------------------------------------------------------- cross-workgroup data
// Loads and stores of the layout data that other workgroups of the same kernel produce or consume
// (the decomposed single-launch layer). With C set they are device-scope accesses: sc1 loads and
// stores, which the AMDGPU memory model uses for relaxed agent-scope atomics and which need no
// cache write-back or invalidation; without it, plain accesses (a kernel boundary orders them).
template <bool C>
__device__ __forceinline__ int32_t ld32(const int32_t* p) {
  if constexpr (C)
    return __hip_atomic_load(const_cast<int32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    return *p;
}
template <bool C>
__device__ __forceinline__ uint32_t ld32(const uint32_t* p) {
  if constexpr (C)
    return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    return *p;
}
template <bool C, class T>
__device__ __forceinline__ void st32(T* p, T v) {
  if constexpr (C)
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    *p = v;
}

// ---------------------------------------------------------------- launchers (host side)
size_t single_lds_bytes(const Geom& g);
bool layout_single(const Geom& g);  // true if epl_layout runs as one launch for this geometry
// K1 and K2 only: histograms, dedup masks and the prefix scans, left in the workspace for a
// finalize step (route_finalize_kernel, or the fused finalize in the dispatch kernels).
hipError_t launch_layout_counts(const Geom& g, const int32_t* idx, int32_t* ws, int32_t* send_cnt, int32_t* rank_cnt,
                                int32_t* tok_nranks, int32_t* num_invalid, hipStream_t stream);
// K3 only, after launch_layout_counts on the same stream.
hipError_t launch_layout_finalize(const Geom& g, const int32_t* idx, int32_t* ws, int32_t* expert_off,
                                  int32_t* rank_off, int32_t* seg_off, int32_t* pair_row, int32_t* pair_rslot,
                                  int32_t* recv_src, int32_t* recv_j, hipStream_t stream);
hipError_t launch_layout(const Geom& g, const int32_t* idx, int32_t* ws, int32_t* send_cnt, int32_t* rank_cnt,
                         int32_t* expert_off, int32_t* rank_off, int32_t* seg_off, int32_t* tok_nranks,
                         int32_t* pair_row, int32_t* pair_rslot, int32_t* recv_src, int32_t* recv_j,
                         int32_t* num_invalid, hipStream_t stream);

// pitch: elements from one recv row to the next (>= H, a multiple of 64).
hipError_t launch_dispatch_bf16(const void* x, const int32_t* pair_row, void* recv, int64_t T, int k, int H,
                                int pitch, int64_t cap, hipStream_t stream);
hipError_t launch_dispatch_fp8(const void* x, const int32_t* pair_row, void* recv, float* recv_scale, int64_t T,
                               int k, int H, int pitch, int64_t cap, hipStream_t stream);
// The layout's finalize step fused into the bf16 dispatch (after launch_layout_counts on the same
// stream), for the geometries fused_dispatch_ok accepts.
bool fused_dispatch_ok(const Geom& g, bool fp8);
hipError_t launch_fused_dispatch(const Geom& g, const int32_t* idx, int32_t* ws, int32_t* expert_off,
                                 int32_t* rank_off, int32_t* seg_off, int32_t* pair_row, int32_t* pair_rslot,
                                 int32_t* recv_src, int32_t* recv_j, const void* x, void* recv, int H, int pitch,
                                 int64_t cap, hipStream_t stream);
// The decomposed single-launch layout and dispatch (bf16, the geometries fused_dispatch_ok
// accepts). count_groups 0 picks the default split; spin_ticks bounds every wait (100 MHz ticks);
// ready_target is the published value the send workgroups wait for (1; a test passes 2 to force a
// give-up). wait_status receives 0, or the give-up bits, when the launch completes.
struct DecomposedOpts {
  int count_groups;
  int64_t spin_ticks;
  int ready_target;
};
// Workgroups of the launch by role, and the device's co-resident capacity for it.
struct DecomposedPlan {
  int grid, count_groups, send_groups, combine_groups, capacity;
};
// How the layer variants' combine workgroups learn that a row chunk has arrived (Data-as-Flag):
// kDafNone is the launch without combine workgroups (layout and dispatch only).
constexpr int kDafNone = 0;       // no combine role
constexpr int kDafSentinel = 1;   // Sentinel Polling: every element compared with the reserved pattern
constexpr int kDafFlag = 2;       // Token-Flag Fusion: an epoch flag per 1 KiB chunk, stored after the chunk
constexpr int kDafChecksum = 3;   // Data-for-Checksum: a salted hash per 1 KiB chunk, checked against the data
hipError_t plan_decomposed(const Geom& g, int H, int count_groups, int sync, DecomposedPlan* plan);
// sync != kDafNone: the layer variant, whose combine workgroups gather the rows into out with the
// weights topk_w as the send workgroups write them; marks and epoch serve kDafFlag and kDafChecksum.
hipError_t launch_decomposed(const Geom& g, const int32_t* idx, int32_t* ws, const epl_layout_buffers& L,
                             const void* x, void* recv, int H, int pitch, int64_t cap, const DecomposedOpts& opts,
                             int32_t* wait_status, hipStream_t stream, int sync = kDafNone,
                             const float* topk_w = nullptr, void* out = nullptr, uint64_t* marks = nullptr,
                             uint64_t epoch = 0);
// Every 16-byte vector of buf [nvec] set to the bf16 sentinel.
hipError_t launch_sentinel_fill(void* buf, int64_t nvec, hipStream_t stream);
// y rows are pitch elements apart.
hipError_t launch_combine(const void* y, const float* w, const int32_t* pair_row, void* out, int64_t T, int k,
                          int H, int pitch, hipStream_t stream);

hipError_t launch_locate_rows(const int32_t* expert_off, const int32_t* rows, int64_t n, int E, int32_t* expert,
                              int32_t* offset, hipStream_t stream);
hipError_t launch_hop_schedule(const int32_t* send_cnt, const int32_t* order, const int32_t* hop, int R, int E,
                               int rows, int n, int NH, int32_t* start_expert, int32_t* start_offset,
                               int32_t* class_cnt, hipStream_t stream);
// recv_scale non-null: fp8 payload (rows quantised as in launch_dispatch_fp8).
hipError_t launch_dispatch_scheduled(const void* x, const int32_t* send_cnt, const int32_t* seg_off,
                                     const int32_t* recv_src, void* recv, float* recv_scale, int R, int E, int rows,
                                     int n, int64_t T, int k, int H, int pitch, int64_t cap, hipStream_t stream);
hipError_t launch_debug_e4m3(const float* in, uint8_t* out, int64_t n, hipStream_t stream);
hipError_t launch_debug_bf16(const float* in, uint16_t* out, int64_t n, hipStream_t stream);

}  // namespace epl
