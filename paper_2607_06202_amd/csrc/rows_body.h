// Device bodies of the row kernels that place each token's pairs as they send them, shared by
// the fused finalize-and-send kernel (dispatch.hip) and the decomposed single-launch layer
// (decomposed.hip), where they read the layout data other workgroups of the same kernel wrote
// with device-scope loads (the C template argument, see ld32).
#pragma once

#include "epl_internal.h"

namespace epl {

constexpr int kDispatchThreads = 256;  // the fused kernel (its metadata workgroups scan with layout-sized blocks)
constexpr int kWavesPerBlock = kDispatchThreads / kWave;
// Workgroup sizes of the plain kernels. Whole layer, two runs each, dispatch us with 128 / 256 /
// 512 threads: decode (bf16) 183.4-183.6 / 177.7-178.0 / 178.6-179.2; EP=256 (bf16) 396.8-397.1 /
// 375.8-376.2 / 389.0-389.3; prefill (bf16) 3327 / 3239-3243 / 3282-3284; skewed fp8 202.3-203.2 /
// 205.3-205.4 / 228.6.
constexpr int kPlainThreads = 256;     // the plain bf16 dispatch kernel
constexpr int kPlainWaves = kPlainThreads / kWave;
constexpr int kFp8Threads = 128;       // the fp8 dispatch kernel
constexpr int kFp8Waves = kFp8Threads / kWave;
// bf16 work unit: one token's columns [u*kBf16Cols, (u+1)*kBf16Cols) in 16-byte vectors.
constexpr int kBf16VPL = 4;                     // vectors per lane in one unit
constexpr int kBf16Cols = kWave * kBf16VPL;     // 256 vectors = 4 KiB of a row
constexpr int64_t kBufferLoadXBytes = 200ll << 20;  // x at least this large: buffer loads (see dispatch_bf16_unit)

// Store one 16-byte vector at vector index v of a row of nv vectors through a buffer resource
// scoped to that row, with an explicit cache policy. The resource bounds (nv * 16 bytes) also
// guard the row. Measured on MI355X, layout -> dispatch -> combine back to back:
// * bf16 rows: sc1 beat default-policy stores (decode 175 against 179 us). Nontemporal stores
//   were slower at every size: about +40 us at decode and EP=256, +105 us at prefill.
// * fp8 rows: sc1+nt beat both (skewed fp8 EP=64: 207 us, against 246 us with sc1 and 252 us
//   with default stores). The fp8 scales are partial-line writes of 32 bytes per row and pass;
//   for them plain stores measured faster than nontemporal ones (235 -> 230 us).
template <int POLICY>
__device__ __forceinline__ void store_row_policy(u32x4 val, u32x4* row_base, int nv, int v) {
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(row_base, 0, nv * 16, kBufferRsrcWord3);
  __builtin_amdgcn_raw_buffer_store_b128(val, rsrc, v * 16, 0, POLICY);
}

// bf16: unit = (token g, column chunk c). The wave loads its chunk of x[g] once and stores it
// to the k destination rows, interleaving destinations per vector. x rows are nv vectors apart,
// recv rows pv (the receive pitch in 16-byte vectors).
//
// BUF_X selects how x is read, both with the default cache policy: buffer loads through a
// resource bounded to the row, or plain global loads. Measured over three repetitions each
// (dispatch alone, x rotated):
// * EP=32 prefill: 3293 -> 3252 us with buffer loads;
// * EP=256: 380.5 -> 376.3 us with buffer loads;
// * EP=64 decode: 176.4 -> 178.1 us, slower with buffer loads.
// The launcher takes buffer loads for an x of 200 MB or more, a threshold between decode's 117 MB
// and the 235 MB and 1.9 GB of the others; why the instruction form matters is not established.
// row_of() returns, in lane j < k, the packed row of pair j (-1 if invalid); it is called after the
// loads of x are issued, so whatever it loads is in flight together with them. An inactive wave
// loads and calls row_of() (which may hold a workgroup barrier) but stores nothing. check(buf, on)
// sees the unit's loaded vectors (on[u]: vector u lies inside the row) before they are stored, and
// after(buf, on, my_row) runs once they are issued (my_row: lane j's packed row, as above).
struct NoCheck {
  __device__ __forceinline__ void operator()(const u32x4*, const bool*) const {}
};
struct NoAfter {
  __device__ __forceinline__ void operator()(const u32x4*, const bool*, int) const {}
};
template <bool BUF_X, class RowFn, class CheckFn = NoCheck, class AfterFn = NoAfter>
__device__ __forceinline__ void dispatch_bf16_unit(const u32x4* __restrict__ x, RowFn row_of, u32x4* __restrict__ recv,
                                                   int64_t g, int c, int k, int nv, int pv, int64_t cap, int lane,
                                                   bool active = true, CheckFn check = CheckFn(),
                                                   AfterFn after = AfterFn()) {
  const u32x4* xr = x + g * nv;
  const int v0 = c * kBf16Cols + lane;
  // Loads are unconditional (index clamped into the row) so that all of them are in flight
  // together; only the stores are guarded. Default cache policy: it measured faster than
  // nontemporal loads here, though x is read once.
  u32x4 buf[kBf16VPL];
  if constexpr (BUF_X) {
    const __amdgpu_buffer_rsrc_t xs = __builtin_amdgcn_make_buffer_rsrc(const_cast<u32x4*>(xr), 0, nv * 16, kBufferRsrcWord3);
#pragma unroll
    for (int u = 0; u < kBf16VPL; ++u) buf[u] = __builtin_amdgcn_raw_buffer_load_b128(xs, min(v0 + u * kWave, nv - 1) * 16, 0, 0);
  } else {
#pragma unroll
    for (int u = 0; u < kBf16VPL; ++u) buf[u] = xr[min(v0 + u * kWave, nv - 1)];
  }
  const int my_row = row_of();
  if (!active) return;
  bool on[kBf16VPL];
#pragma unroll
  for (int u = 0; u < kBf16VPL; ++u) on[u] = v0 + u * kWave < nv;
  check(buf, on);
#pragma unroll
  for (int u = 0; u < kBf16VPL; ++u) {
    const int v = v0 + u * kWave;
    for (int j = 0; j < k; ++j) {
      const int row = __builtin_amdgcn_readlane(my_row, j);
      if (row < 0 || row >= cap) continue;
      if (v < nv) store_row_policy<kCachePolicySc1>(buf[u], recv + (int64_t)row * pv, nv, v);
    }
  }
  after(buf, on, my_row);
}

// fp8: unit = (token g, pass p) covering elements [1024p, 1024p + 1024). Lane l quantises
// elements [16l, 16l+16) of the pass: two 16-byte bf16 loads -> one 16-byte E4M3 store per
// destination. A 128-element block spans 8 lanes, whose max is combined with three
// xor-shuffles; the first lane of each block stores that block's scale for every destination.
// recv rows are pq 16-byte vectors apart (the receive pitch, in bytes / 16).
template <class RowFn>
__device__ __forceinline__ void dispatch_fp8_unit(const u32x4* __restrict__ x, RowFn row_of, u32x4* __restrict__ recv,
                                                  float* __restrict__ recv_scale, int64_t g, int p, int k, int H,
                                                  int pq, int64_t cap, int lane) {
  const int NB = H / 128;
  const int nvq = H / 16;  // 16-byte fp8 vectors per row
  const u32x4* xr = x + g * (H / 8);
  const int vq = p * kWave + lane;  // fp8 vector index = element / 16
  const bool on = vq < nvq;         // whole 8-lane blocks are on or off (H % 128 == 0)
  const int vl = min(vq, nvq - 1);  // clamped so the loads need no branch
  u32x4 a = xr[2 * vl];
  u32x4 bv = xr[2 * vl + 1];
  const int my_row = row_of();
  if (!on) a = bv = u32x4{0, 0, 0, 0};
  float f[16];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = bf16lo_to_f32(a[i]);
    f[2 * i + 1] = bf16hi_to_f32(a[i]);
    f[8 + 2 * i] = bf16lo_to_f32(bv[i]);
    f[8 + 2 * i + 1] = bf16hi_to_f32(bv[i]);
  }
  float amax = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) amax = fmaxf(amax, fabsf(f[i]));
  amax = fmaxf(amax, __shfl_xor(amax, 1, kWave));
  amax = fmaxf(amax, __shfl_xor(amax, 2, kWave));
  amax = fmaxf(amax, __shfl_xor(amax, 4, kWave));
  const float s = amax / 448.0f;
  u32x4 q = {0, 0, 0, 0};
  if (amax != 0.0f) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      q[i] = f32x4_to_e4m3x4(f[4 * i] / s, f[4 * i + 1] / s, f[4 * i + 2] / s, f[4 * i + 3] / s);
  }
  const bool scale_lane = on && (lane % 8) == 0;
  for (int j = 0; j < k; ++j) {
    const int row = __builtin_amdgcn_readlane(my_row, j);
    if (row < 0 || row >= cap) continue;
    if (on) store_row_policy<kCachePolicySc1Nt>(q, recv + (int64_t)row * pq, nvq, vq);
    if (scale_lane) recv_scale[(int64_t)row * NB + vq / 8] = s;
  }
}

struct FusedLayout {
  Geom G;
  const int32_t* idx;
  const int32_t* chunk_e;   // [E][nblk] rows of each expert before each chunk (K2)
  const int32_t* chunk_r;   // [nblk][R] slots of each rank before each chunk (K2)
  const int32_t* recv_cnt;  // [E]
  const int32_t* seg_rel;   // [E][R]
  const uint32_t* fmask;    // [T] first-pair bitmask of each token (K1)
  int32_t* expert_off;
  int32_t* rank_off;
  int32_t* seg_off;
  int32_t* pair_row;
  int32_t* pair_rslot;
  int32_t* recv_src;
  int32_t* recv_j;
};

// Sizes the fused kernel is built for: at most kFusedSlots * 64 pairs per chunk (CT * k) and
// kFusedPer * 64 experts. hist is this wave's LDS [E + R].
constexpr int kFusedSlots = 4;
constexpr int kFusedPer = 4;
template <bool C>
__device__ __forceinline__ int token_rows(const FusedLayout& F, int64_t g, bool meta, int32_t* hist, int lane) {
  const Geom& G = F.G;
  const int k = G.k;
  const int s = (int)(g / G.Tr);
  const int t = (int)(g - (int64_t)s * G.Tr);
  const int c = t / G.CT;
  const int b = s * G.NC + c;
  const int64_t tok0 = (int64_t)s * G.Tr + (int64_t)c * G.CT;  // first token of the chunk
  const int nb = (int)(g - tok0) * k;                            // earlier pairs of the chunk, < CT * k
  const int64_t cb = tok0 * k;

  // Every independent load first (indices clamped, so none sits behind a branch).
  const bool mine = lane < k;
  const int e = F.idx[g * k + min(lane, k - 1)];
  const uint32_t fm = ld32<C>(&F.fmask[g]);
  const int per = (G.E + kWave - 1) / kWave;  // experts per lane in the prefix of recv_cnt, <= kFusedPer
  int rc[kFusedPer];
#pragma unroll
  for (int i = 0; i < kFusedPer; ++i) rc[i] = ld32<C>(&F.recv_cnt[min(lane * per + i, G.E - 1)]);
  int ep[kFusedSlots];
  uint32_t fp[kFusedSlots];
#pragma unroll
  for (int q = 0; q < kFusedSlots; ++q) {
    const int i = min(q * kWave + lane, max(nb - 1, 0));
    ep[q] = nb > 0 ? F.idx[cb + i] : -1;
    fp[q] = nb > 0 ? ld32<C>(&F.fmask[tok0 + small_div(i, G.inv_k)]) : 0u;
  }
  const bool valid = mine && (unsigned)e < (unsigned)G.E;
  const int ev = valid ? e : 0;
  const int d = valid ? small_div(e, G.inv_El) : 0;
  const int base_e = ld32<C>(&F.chunk_e[(int64_t)ev * G.nblk + b]);
  const int base_r = ld32<C>(&F.chunk_r[(int64_t)b * G.R + d]);

  // Histograms of the chunk's earlier pairs: experts, and ranks of first pairs.
  int32_t* he = hist;
  int32_t* hr = hist + G.E;
  for (int i = lane; i < G.E + G.R; i += kWave) hist[i] = 0;
#pragma unroll
  for (int q = 0; q < kFusedSlots; ++q) {
    const int i = q * kWave + lane;
    const int xe = ep[q];
    if (i < nb && (unsigned)xe < (unsigned)G.E) {
      atomicAdd(&he[xe], 1);
      const int tp = small_div(i, G.inv_k);
      if ((fp[q] >> (i - tp * k)) & 1u) atomicAdd(&hr[small_div(xe, G.inv_El)], 1);
    }
  }

  // First row of each expert: exclusive prefix of recv_cnt. Lane L holds experts
  // [L*per, L*per + per); the prefix at expert ev comes from lane ev / per.
  int run = 0;
  int ps[kFusedPer];
#pragma unroll
  for (int i = 0; i < kFusedPer; ++i) {
    run += (i < per && lane * per + i < G.E) ? rc[i] : 0;
    ps[i] = run;
  }
  const int incl = wave_inclusive_sum(run);
  const int P = __shfl(incl, kWave - 1, kWave);  // valid pairs in the whole layout
  const int L = ev / per;
  const int il = ev - L * per;
  int eoff = __shfl(incl - run, L, kWave);
#pragma unroll
  for (int i = 0; i + 1 < kFusedPer; ++i) {
    if (i + 1 >= per) break;  // wave-uniform
    const int v = __shfl(ps[i], L, kWave);
    if (i == il - 1) eoff += v;
  }

  const int rank_e = he[ev] + rank_in_mask(match_key(valid, ev, G.ebits));
  const bool first = valid && ((fm >> min(lane, 31)) & 1u);
  const int row = valid ? eoff + base_e + rank_e : -1;
  const int slot = first ? base_r + hr[d] : -1;
  // The token's first pair on a rank is its lowest valid lane with that rank.
  const uint64_t md = match_key(valid, d, G.rbits);
  const int lead = valid ? (int)__builtin_ctzll(md) : 0;
  const int rslot = __shfl(slot, lead, kWave);
  if (meta && mine) {
    F.pair_row[g * k + lane] = row;
    F.pair_rslot[g * k + lane] = valid ? rslot : -1;
    if (valid && row < P) {  // always true for a consistent layout; keeps stores in bounds
      F.recv_src[row] = (int32_t)g;
      F.recv_j[row] = lane;
    }
  }
  return mine ? row : -1;
}

// Workgroups past the dispatch units: expert_off and rank_off (the first of them) and one slice
// of seg_off each. lds holds at least E + 1 ints.
template <bool C>
__device__ __forceinline__ void fused_meta_block(const FusedLayout& F, int m, int nmeta, int32_t* lds) {
  static_assert(kDispatchThreads == kLayoutThreads, "block_exclusive_sum assumes layout-sized workgroups");
  __shared__ int32_t scratch[kLayoutWaves];
  const Geom& G = F.G;
  const int tid = threadIdx.x;
  int32_t* eoff = lds;
  const int per = (G.E + kLayoutThreads - 1) / kLayoutThreads;
  const int e0 = min(G.E, tid * per), e1 = min(G.E, e0 + per);
  int rc[kLayoutSlots];
#pragma unroll
  for (int q = 0; q < kLayoutSlots; ++q) rc[q] = ld32<C>(&F.recv_cnt[min(e0 + q, G.E - 1)]);
  int sum = 0;
#pragma unroll
  for (int q = 0; q < kLayoutSlots; ++q) sum += e0 + q < e1 ? rc[q] : 0;
  int total;
  int run = block_exclusive_sum(sum, total, scratch);  // synchronises the workgroup
#pragma unroll
  for (int q = 0; q < kLayoutSlots; ++q) {
    if (e0 + q >= e1) break;
    eoff[e0 + q] = run;
    run += rc[q];
  }
  if (tid == 0) eoff[G.E] = total;
  __syncthreads();
  if (m == 0) {
    for (int e = tid; e <= G.E; e += kLayoutThreads) F.expert_off[e] = eoff[e];
    for (int r = tid; r <= G.R; r += kLayoutThreads) F.rank_off[r] = eoff[r * G.El];
  }
  const int nseg = G.E * G.R;
  const int seg_per = (nseg + nmeta - 1) / nmeta;
  const int i1 = min(nseg, (m + 1) * seg_per);
  for (int i = m * seg_per + tid; i < i1; i += kLayoutThreads)
    F.seg_off[i] = eoff[small_div(i, G.inv_R)] + ld32<C>(&F.seg_rel[i]);
}

}  // namespace epl
