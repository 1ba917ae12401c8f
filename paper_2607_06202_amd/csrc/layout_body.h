// Device bodies of the layout's counting kernels, shared by the three-launch layout
// (layout.hip: K1 route_hist, K2 route_scan) and the decomposed single-launch layer
// (decomposed.hip), where count workgroups run the same bodies with device-scope accesses to the
// data other workgroups of the same kernel read (the C template argument, see ld32/st32).
#pragma once

#include "epl_internal.h"

namespace epl {

// Dedup of one token: bit j is set if pair j is valid (dt[j] >= 0) and no earlier valid pair of
// the token targets the same destination rank dt[j].
__device__ __forceinline__ uint32_t first_rank_mask(const int32_t* dt, int k) {
  uint32_t mask = 0;
  for (int j = 0; j < k; ++j) {
    const int d = dt[j];
    if (d < 0) continue;
    bool first = true;
    for (int jj = 0; jj < j; ++jj) first &= (dt[jj] != d);
    if (first) mask |= 1u << j;
  }
  return mask;
}

// Workgroups are dealt to the MI355X's 8 XCDs in turn (workgroup i to XCD i % 8), and each XCD
// has its own L2. K1 and K3 take chunk xcd_chunk(i, nblk) in workgroup i, so that every XCD
// handles one contiguous eighth of the chunks (the tail past 8 * (nblk / 8) keeps i). Their
// small scattered stores then fall into whole lines in one L2: K1's per-chunk expert counts
// ([E][nblk], adjacent chunks adjacent), and K3's recv_src / recv_j (within an expert, the rows
// of adjacent chunks of a source rank are adjacent).
constexpr int kXcds = 8;
__device__ __forceinline__ int xcd_chunk(int i, int n) {
  const int per = n / kXcds;
  return i < per * kXcds ? (i % kXcds) * per + i / kXcds : i;
}

// K1 on chunk b (CT whole tokens of one source rank): LDS histograms of expert ids and of
// first-per-token destination ranks, the per-token first-pair bitmask, tok_nranks, the chunk's
// invalid count, the chunk's row of chunk_r [nblk][R], and its expert counts: the chunk's column
// of chunk_e [E][nblk] without C; with C, the chunk's row of cnt [nblk][E] (device-scope stores
// of whole lines; single 4-byte device-scope stores into lines other workgroups also write each
// cost a read-modify-write of the line in memory). lds holds E + R + kMaxChunkPairs ints, red
// kLayoutWaves; the whole workgroup calls it.
template <bool C>
__device__ __forceinline__ void hist_chunk(const Geom& G, int b, const int32_t* __restrict__ idx,
                                           int32_t* __restrict__ tok_nranks, int32_t* __restrict__ chunk_e,
                                           int32_t* __restrict__ chunk_r, int32_t* __restrict__ inval,
                                           uint32_t* __restrict__ fmask, int32_t* lds, int32_t* red,
                                           int32_t* __restrict__ cnt = nullptr) {
  int32_t* hist_e = lds;           // [E]
  int32_t* hist_r = hist_e + G.E;  // [R]
  int32_t* dst = hist_r + G.R;     // [kMaxChunkPairs] destination rank of each pair, -1 if invalid

  const int tid = threadIdx.x;
  const int s = b / G.NC;
  const int c = b - s * G.NC;
  const int t0 = c * G.CT;
  const int nt = max(0, min(G.CT, G.Tr - t0));
  const int np = nt * G.k;
  const int64_t g0 = (int64_t)s * G.Tr + t0;

  // Issue the global loads first; their latency overlaps the LDS clearing and the barrier.
  const int32_t* src = idx + g0 * G.k;
  int ids[kChunkSlots];
#pragma unroll
  for (int q = 0; q < kChunkSlots; ++q) {
    const int i = tid + q * kLayoutThreads;
    ids[q] = i < np ? src[i] : 0;
  }
  for (int i = tid; i < G.E + G.R; i += kLayoutThreads) lds[i] = 0;
  __syncthreads();

  int my_inval = 0;
#pragma unroll
  for (int q = 0; q < kChunkSlots; ++q) {
    const int i = tid + q * kLayoutThreads;
    if (i >= np) break;
    const int e = ids[q];
    const bool ok = (unsigned)e < (unsigned)G.E;
    dst[i] = ok ? small_div(e, G.inv_El) : -1;
    if (ok)
      atomicAdd(&hist_e[e], 1);
    else
      ++my_inval;
  }
  __syncthreads();

  // Dedup: a pair is the first of its token for its destination rank if no earlier valid pair
  // of the token targets the same rank. One thread per token.
  for (int t = tid; t < nt; t += kLayoutThreads) {
    const int32_t* dt = dst + t * G.k;
    const uint32_t mask = first_rank_mask(dt, G.k);
    for (uint32_t m = mask; m; m &= m - 1) atomicAdd(&hist_r[dt[__builtin_ctz(m)]], 1);
    tok_nranks[g0 + t] = __popc(mask);
    st32<C>(&fmask[g0 + t], mask);
  }

  const int wsum = wave_sum(my_inval);
  if (lane_id() == 0) red[tid / kWave] = wsum;
  __syncthreads();

  if constexpr (C)
    for (int e = tid; e < G.E; e += kLayoutThreads) st32<C>(&cnt[(int64_t)b * G.E + e], hist_e[e]);
  else
    for (int e = tid; e < G.E; e += kLayoutThreads) chunk_e[(int64_t)e * G.nblk + b] = hist_e[e];
  for (int r = tid; r < G.R; r += kLayoutThreads) st32<C>(&chunk_r[(int64_t)b * G.R + r], hist_r[r]);
  if (tid == 0) {
    int n = 0;
    for (int w = 0; w < kLayoutWaves; ++w) n += red[w];
    st32<C>(&inval[b], n);
  }
}

constexpr int kScanV = 4;  // consecutive elements per thread in one workgroup scan step

// K2 item b of E + R + 1: expert column b < E, source rank b - E < R, or the invalid total.
// scratch holds kLayoutWaves ints, seg_start EPL_MAX_EXPERTS + 1; the whole workgroup calls it.
template <bool C>
__device__ __forceinline__ void scan_item(const Geom& G, int b, int32_t* __restrict__ chunk_e,
                                          int32_t* __restrict__ chunk_r, const int32_t* __restrict__ inval,
                                          int32_t* __restrict__ recv_cnt, int32_t* __restrict__ send_cnt,
                                          int32_t* __restrict__ rank_cnt, int32_t* __restrict__ seg_rel,
                                          int32_t* __restrict__ num_invalid, int32_t* scratch, int32_t* seg_start,
                                          const int32_t* __restrict__ cnt = nullptr) {
  const int tid = threadIdx.x;
  if (b < G.E) {
    // Expert column e, laid out [source rank][chunk] (flat index s * NC + c, the order of the
    // expert's rows): an exclusive scan over the whole column gives each chunk's rows relative to
    // the expert start. The workgroup scans kScanV consecutive chunks per thread at a time; the
    // value at each rank's first chunk is that rank's segment start.
    const int e = b;
    int32_t* col = chunk_e + (int64_t)e * G.nblk;
    int carry = 0;
    for (int base = 0; base < G.nblk; base += kLayoutThreads * kScanV) {
      const int b0 = base + tid * kScanV;
      int h[kScanV];
      int sum = 0;
#pragma unroll
      for (int v = 0; v < kScanV; ++v) {
        // With C the counts come from cnt [nblk][E] (K1's rows); the bases go to chunk_e either way.
        if constexpr (C)
          h[v] = b0 + v < G.nblk ? ld32<C>(&cnt[(int64_t)(b0 + v) * G.E + e]) : 0;
        else
          h[v] = b0 + v < G.nblk ? col[b0 + v] : 0;
        sum += h[v];
      }
      int total;
      int run = carry + block_exclusive_sum(sum, total, scratch);
#pragma unroll
      for (int v = 0; v < kScanV; ++v) {
        const int bb = b0 + v;
        if (bb < G.nblk) {
          st32<C>(&col[bb], run);
          const int s = bb / G.NC;
          if (bb == s * G.NC) seg_start[s] = run;
        }
        run += h[v];
      }
      carry += total;
    }
    if (tid == 0) seg_start[G.R] = carry;
    __syncthreads();
    for (int s = tid; s < G.R; s += kLayoutThreads) {
      st32<C>(&seg_rel[e * G.R + s], seg_start[s]);
      send_cnt[s * G.E + e] = seg_start[s + 1] - seg_start[s];
    }
    if (tid == 0) st32<C>(&recv_cnt[e], carry);
  } else if (b < G.E + G.R) {
    // Source rank s: per destination rank r, slots of earlier chunks come first. The rank's
    // [chunk][R] block of counts is scanned as one flat sequence in (r, chunk) order, so each r
    // is a contiguous segment; an element's slot base is the flat exclusive prefix minus the
    // prefix at its segment's first chunk.
    const int s = b - G.E;
    int32_t* rows = chunk_r + (int64_t)s * G.NC * G.R;  // this rank's NC chunk rows of R counts
    const int n = G.NC * G.R;
    int carry = 0;
    for (int base = 0; base < n; base += kLayoutThreads * kScanV) {
      int h[kScanV], at[kScanV], rr[kScanV];
      int sum = 0;
#pragma unroll
      for (int v = 0; v < kScanV; ++v) {
        const int f = base + tid * kScanV + v;
        rr[v] = f / G.NC;
        const int c = f - rr[v] * G.NC;
        at[v] = f < n ? c * G.R + rr[v] : -1;
        h[v] = f < n ? ld32<C>(&rows[at[v]]) : 0;
        sum += h[v];
      }
      int total;
      int run = carry + block_exclusive_sum(sum, total, scratch);
      int pre[kScanV];
#pragma unroll
      for (int v = 0; v < kScanV; ++v) {
        pre[v] = run;
        if (at[v] >= 0 && at[v] < G.R) seg_start[rr[v]] = run;  // chunk 0 of rank rr[v]
        run += h[v];
      }
      carry += total;
      __syncthreads();  // segment starts found in this step are visible
#pragma unroll
      for (int v = 0; v < kScanV; ++v)
        if (at[v] >= 0) st32<C>(&rows[at[v]], pre[v] - seg_start[rr[v]]);
    }
    if (tid == 0) seg_start[G.R] = carry;
    __syncthreads();
    for (int r = tid; r < G.R; r += kLayoutThreads) rank_cnt[s * G.R + r] = seg_start[r + 1] - seg_start[r];
  } else {
    int n = 0;
    for (int i = tid; i < G.nblk; i += kLayoutThreads) n += ld32<C>(&inval[i]);
    const int w = wave_sum(n);
    if (lane_id() == 0) scratch[tid / kWave] = w;
    __syncthreads();
    if (tid == 0) {
      int t = 0;
      for (int i = 0; i < kLayoutWaves; ++i) t += scratch[i];
      num_invalid[0] = t;
    }
  }
}

}  // namespace epl
