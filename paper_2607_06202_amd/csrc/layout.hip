// Routing layout for MoE dispatch on one GPU: per-(source rank, expert) histograms, CalCumSum
// prefix scans, stable packed-row assignment and per-token destination-rank dedup.
//
// The paper's dispatch reports per-expert token counts from every source. Prefix sums of those
// counts give each expert's HBM offsets, and tokens are then laid out contiguously per expert
// (Background phases 3 and 5; Kernel Decomposition: TokenCnt-Sending, CalCumSum,
// Token-Reordering). All ranks are virtual here, so the count "exchange" is just reading the
// [rank][expert] matrix by column.
//
// Three launches, no atomics that decide an order, bit-identical on every run (small layouts
// take one launch instead, route_single below, with the same outputs):
//   K1 route_hist      one workgroup per chunk (CT whole tokens of one source rank): LDS
//                      histograms of expert ids and of first-per-token destination ranks, the
//                      per-token first-pair bitmask, tok_nranks and the invalid count.
//   K2 route_scan      one workgroup per expert column: scan over (source rank, chunk) giving
//                      segment offsets relative to the expert start, send_cnt, recv_cnt and
//                      per-chunk base rows. One workgroup per source rank: scan of rank slots
//                      over chunks. One workgroup: num_invalid.
//   K3 route_finalize  one workgroup per chunk: expert_off via an LDS scan of recv_cnt. Each
//                      wave takes a contiguous quarter of the chunk's pairs and gives every pair
//                      its stable rank among equal keys: ballot match over the key bits,
//                      popcount of the lanes below, per-wave LDS running counts. A cross-wave
//                      prefix then yields pair_row, recv_src, recv_j and pair_rslot.
// For bf16 decode-sized layouts epl_layout_dispatch skips K3: the dispatch kernel derives each
// token's rows from K1 and K2's workspace with the same definitions (dispatch.hip).
//
// Small integer quotients (pair -> token within a chunk, expert -> rank, seg_off index -> expert;
// every numerator < 2^21) use small_div, which is exact in that range.
#include "layout_body.h"

namespace epl {

// ------------------------------------------------------------------------------------ K1
__global__ void __launch_bounds__(kLayoutThreads)
    route_hist_kernel(Geom G, const int32_t* __restrict__ idx, int32_t* __restrict__ tok_nranks,
                      int32_t* __restrict__ chunk_e, int32_t* __restrict__ chunk_r, int32_t* __restrict__ inval,
                      uint32_t* __restrict__ fmask) {
  extern __shared__ int32_t lds[];
  __shared__ int32_t red[kLayoutWaves];
  hist_chunk<false>(G, xcd_chunk(blockIdx.x, G.nblk), idx, tok_nranks, chunk_e, chunk_r, inval, fmask, lds, red);
}

// ------------------------------------------------------------------------------------ K2
__global__ void __launch_bounds__(kLayoutThreads)
    route_scan_kernel(Geom G, int32_t* __restrict__ chunk_e, int32_t* __restrict__ chunk_r,
                      const int32_t* __restrict__ inval, int32_t* __restrict__ recv_cnt, int32_t* __restrict__ send_cnt,
                      int32_t* __restrict__ rank_cnt, int32_t* __restrict__ seg_rel, int32_t* __restrict__ num_invalid) {
  __shared__ int32_t scratch[kLayoutWaves];
  __shared__ int32_t seg_start[EPL_MAX_EXPERTS + 1];  // per source rank (R <= E), then the total
  scan_item<false>(G, blockIdx.x, chunk_e, chunk_r, inval, recv_cnt, send_cnt, rank_cnt, seg_rel, num_invalid,
                   scratch, seg_start);
}

// Rows and rank slots for the pairs of one chunk. All inputs are in LDS:
// * ekey/dkey [np]: expert and destination rank of each pair, -1 if invalid;
// * fm [nt]: each token's first-pair-per-rank bitmask;
// * base_e [E]: the first packed row of this chunk's pairs of expert e;
// * base_r [R]: the first slot of this chunk's tokens bound for rank r;
// * whe/whr [W][E] and [W][R]: zeroed.
// Every pair gets its stable rank among equal keys of the chunk. Each wave takes a contiguous
// quarter of the chunk's pairs: ballot match over the key bits, popcount of the lanes below, and
// per-wave LDS running counts. A cross-wave prefix then yields pair_row, recv_src, recv_j and
// pair_rslot. P is the number of valid pairs in the whole layout; rows at or past it are never
// written.
__device__ __forceinline__ void assign_chunk_rows(const Geom& G, int np, int64_t g0, int P,
                                                  const int32_t* ekey, const int32_t* dkey, const uint32_t* fm,
                                                  const int32_t* base_e, const int32_t* base_r, int32_t* whe,
                                                  int32_t* whr, int32_t* rs, int32_t* __restrict__ pair_row,
                                                  int32_t* __restrict__ pair_rslot, int32_t* __restrict__ recv_src,
                                                  int32_t* __restrict__ recv_j) {
  const int tid = threadIdx.x;
  // Stable ranks. Wave w owns pairs [w*Q, w*Q + Q) of the chunk, walked 64 at a time in pair
  // order; whe/whr[w][key] count the keys this wave has already seen.
  const int w = tid / kWave;
  const int lane = tid - w * kWave;
  const int Q = ((np + kLayoutThreads - 1) / kLayoutThreads) * kWave;
  const int p_beg = w * Q;
  const int p_end = min(np, p_beg + Q);
  int rank_e[kChunkSlots], rank_r[kChunkSlots];
#pragma unroll
  for (int it = 0; it < kChunkSlots; ++it) {
    rank_e[it] = 0;
    rank_r[it] = 0;
    if (p_beg + it * kWave >= p_end) continue;  // wave-uniform
    const int p = p_beg + it * kWave + lane;
    const bool active = p < p_end;
    const int e = active ? ekey[p] : -1;
    const int d = active ? dkey[p] : -1;
    const bool valid = e >= 0;
    const int t = small_div(p, G.inv_k);
    const bool first = valid && ((fm[t] >> (p - t * G.k)) & 1u);

    const uint64_t me = match_key(valid, e, G.ebits);
    const int lo_e = rank_in_mask(me);
    const int seen_e = valid ? whe[w * G.E + e] : 0;
    if (valid && lo_e == 0) whe[w * G.E + e] = seen_e + __popcll(me);  // one lane per key
    rank_e[it] = seen_e + lo_e;

    const uint64_t mr = match_key(first, d, G.rbits);
    const int lo_r = rank_in_mask(mr);
    const int seen_r = first ? whr[w * G.R + d] : 0;
    if (first && lo_r == 0) whr[w * G.R + d] = seen_r + __popcll(mr);
    rank_r[it] = seen_r + lo_r;
  }
  __syncthreads();

  // Per-wave counts -> per-wave bases (exclusive prefix over waves, in wave order).
  for (int e = tid; e < G.E; e += kLayoutThreads) {
    int run = 0;
#pragma unroll
    for (int v = 0; v < kLayoutWaves; ++v) {
      const int h = whe[v * G.E + e];
      whe[v * G.E + e] = run;
      run += h;
    }
  }
  for (int r = tid; r < G.R; r += kLayoutThreads) {
    int run = 0;
#pragma unroll
    for (int v = 0; v < kLayoutWaves; ++v) {
      const int h = whr[v * G.R + r];
      whr[v * G.R + r] = run;
      run += h;
    }
  }
  __syncthreads();

#pragma unroll
  for (int it = 0; it < kChunkSlots; ++it) {
    if (p_beg + it * kWave >= p_end) continue;
    const int p = p_beg + it * kWave + lane;
    if (p >= p_end) continue;
    const int e = ekey[p];
    const int t = small_div(p, G.inv_k);
    const int j = p - t * G.k;
    const int64_t g = g0 + t;
    if (e >= 0) {
      const int row = base_e[e] + whe[w * G.E + e] + rank_e[it];
      pair_row[g * G.k + j] = row;
      if (row < P) {  // always true for a consistent layout; keeps stores in bounds
        recv_src[row] = (int32_t)g;
        recv_j[row] = j;
      }
      if ((fm[t] >> j) & 1u) {
        const int d = dkey[p];
        rs[p] = base_r[d] + whr[w * G.R + d] + rank_r[it];
      }
    } else {
      pair_row[g * G.k + j] = -1;
    }
  }
  __syncthreads();

  // Every valid pair reports the slot of its token's first pair on the same rank.
  for (int p = tid; p < np; p += kLayoutThreads) {
    const int d = dkey[p];
    const int t = small_div(p, G.inv_k);
    int slot = -1;
    if (d >= 0) {
      int jf = t * G.k;
      while (dkey[jf] != d) ++jf;
      slot = rs[jf];
    }
    pair_rslot[(g0 + t) * G.k + (p - t * G.k)] = slot;
  }
}

// ------------------------------------------------------------------------------------ K3
__global__ void __launch_bounds__(kLayoutThreads)
    route_finalize_kernel(Geom G, const int32_t* __restrict__ idx, const int32_t* __restrict__ chunk_e,
                          const int32_t* __restrict__ chunk_r, const int32_t* __restrict__ recv_cnt,
                          const int32_t* __restrict__ seg_rel, const uint32_t* __restrict__ fmask,
                          int32_t* __restrict__ expert_off, int32_t* __restrict__ rank_off, int32_t* __restrict__ seg_off,
                          int32_t* __restrict__ pair_row, int32_t* __restrict__ pair_rslot, int32_t* __restrict__ recv_src,
                          int32_t* __restrict__ recv_j) {
  extern __shared__ int32_t lds[];
  int32_t* eoff = lds;                       // [E+1]
  int32_t* base_e = eoff + G.E + 1;          // [E]   first packed row of this chunk's pairs of expert e
  int32_t* base_r = base_e + G.E;            // [R]   first slot of this chunk's tokens bound for rank r
  int32_t* whe = base_r + G.R;               // [W][E] per-wave counts, then per-wave bases
  int32_t* whr = whe + kLayoutWaves * G.E;   // [W][R]
  int32_t* ekey = whr + kLayoutWaves * G.R;  // [kMaxChunkPairs] expert id, -1 invalid
  int32_t* dkey = ekey + kMaxChunkPairs;     // [kMaxChunkPairs] destination rank, -1 invalid
  int32_t* rs = dkey + kMaxChunkPairs;       // [kMaxChunkPairs] slot of first pairs
  uint32_t* fm = reinterpret_cast<uint32_t*>(rs + kMaxChunkPairs);  // [kMaxChunkPairs / 1] token masks
  __shared__ int32_t scratch[kLayoutWaves];

  const int tid = threadIdx.x;
  const int b = xcd_chunk(blockIdx.x, G.nblk);
  const int s = b / G.NC;
  const int c = b - s * G.NC;
  const int t0 = c * G.CT;
  const int nt = max(0, min(G.CT, G.Tr - t0));
  const int np = nt * G.k;
  const int64_t g0 = (int64_t)s * G.Tr + t0;

  // All global inputs of this workgroup are independent: issue them together. That includes
  // the first entries of this workgroup's slice of segment offsets, which are stored at the end.
  const int nseg = G.E * G.R;
  const int seg_per = (nseg + G.nblk - 1) / G.nblk;
  const int seg_i1 = min(nseg, (b + 1) * seg_per);
  constexpr int kSegSlots = 2;
  int seg_pre[kSegSlots];
#pragma unroll
  for (int q = 0; q < kSegSlots; ++q) {
    const int i = b * seg_per + tid + q * kLayoutThreads;
    seg_pre[q] = i < seg_i1 ? seg_rel[i] : 0;
  }
  // Each lane loads its ids, token masks, chunk counts and expert totals into registers first
  // (indices clamped, so no load sits behind a branch), then waits once.
  const int32_t* src = idx + g0 * G.k;
  const int per = (G.E + kLayoutThreads - 1) / kLayoutThreads;  // experts per lane in the scan below
  const int e0 = min(G.E, tid * per), e1 = min(G.E, e0 + per);
  int id_r[kChunkSlots];
  uint32_t fm_r[kChunkSlots];
#pragma unroll
  for (int q = 0; q < kChunkSlots; ++q) {
    id_r[q] = 0;
    fm_r[q] = 0;
  }
  if (np > 0) {  // uniform; idx may be null when there are no tokens
#pragma unroll
    for (int q = 0; q < kChunkSlots; ++q) {
      const int i = tid + q * kLayoutThreads;
      id_r[q] = src[min(i, np - 1)];
      fm_r[q] = fmask[g0 + min(i, nt - 1)];
    }
  }
  int ce_r[kLayoutSlots], cr_r[kLayoutSlots], rc_r[kLayoutSlots];
#pragma unroll
  for (int q = 0; q < kLayoutSlots; ++q) {
    const int e = tid + q * kLayoutThreads;
    ce_r[q] = chunk_e[(int64_t)min(e, G.E - 1) * G.nblk + b];
    cr_r[q] = chunk_r[(int64_t)b * G.R + min(e, G.R - 1)];
    rc_r[q] = recv_cnt[min(e0 + q, G.E - 1)];
  }
  for (int i = tid; i < kLayoutWaves * (G.E + G.R); i += kLayoutThreads) whe[i] = 0;
#pragma unroll
  for (int q = 0; q < kChunkSlots; ++q) {
    const int i = tid + q * kLayoutThreads;
    if (i < np) {
      const int e = id_r[q];
      const bool ok = (unsigned)e < (unsigned)G.E;
      ekey[i] = ok ? e : -1;
      dkey[i] = ok ? small_div(e, G.inv_El) : -1;
    }
    if (i < nt) fm[i] = fm_r[q];
  }
#pragma unroll
  for (int q = 0; q < kLayoutSlots; ++q) {
    const int e = tid + q * kLayoutThreads;
    if (e < G.E) base_e[e] = ce_r[q];
    if (e < G.R) base_r[e] = cr_r[q];
  }

  // expert_off = exclusive scan of recv_cnt; each lane owns the contiguous run [e0, e1).
  {
    int sum = 0;
#pragma unroll
    for (int q = 0; q < kLayoutSlots; ++q) sum += e0 + q < e1 ? rc_r[q] : 0;
    int total;
    int run = block_exclusive_sum(sum, total, scratch);  // synchronises the workgroup
#pragma unroll
    for (int q = 0; q < kLayoutSlots; ++q) {
      if (e0 + q >= e1) break;
      eoff[e0 + q] = run;
      base_e[e0 + q] += run;
      run += rc_r[q];
    }
    if (tid == 0) eoff[G.E] = total;
  }
  __syncthreads();

  assign_chunk_rows(G, np, g0, eoff[G.E], ekey, dkey, fm, base_e, base_r, whe, whr, rs, pair_row, pair_rslot,
                    recv_src, recv_j);

  // Global offsets, off the critical path: block 0 writes expert_off and rank_off; every
  // workgroup rebases one slice of the (expert, source) segment offsets.
  if (b == 0) {
    for (int e = tid; e <= G.E; e += kLayoutThreads) expert_off[e] = eoff[e];
    for (int d = tid; d <= G.R; d += kLayoutThreads) rank_off[d] = eoff[d * G.El];
  }
#pragma unroll
  for (int q = 0; q < kSegSlots; ++q) {
    const int i = b * seg_per + tid + q * kLayoutThreads;
    if (i < seg_i1) seg_off[i] = eoff[small_div(i, G.inv_R)] + seg_pre[q];
  }
  for (int i = b * seg_per + tid + kSegSlots * kLayoutThreads; i < seg_i1; i += kLayoutThreads)
    seg_off[i] = eoff[small_div(i, G.inv_R)] + seg_rel[i];
}

// ------------------------------------------------------------------------------------ single launch
// One launch instead of three, for small layouts (see layout_single). Each workgroup takes one
// chunk, as K1 and K3 do, and recomputes what K1 and K2 would have handed it:
// * a pass over all T*k expert ids fills two LDS histograms, split at the chunk's first pair:
//   the pairs of each expert before the chunk (its row base within the expert, and for the
//   rank's first chunk the seg_off base) and from the chunk on (with the first, the expert totals
//   that give expert_off). The rank's last chunk also counts the rank's own pairs (send_cnt);
// * the dedup of the source rank's earlier tokens gives the chunk's slot base per destination rank.
// The rows are then assigned exactly as in K3. A launch boundary costs several microseconds here;
// the redundant pass is cheaper while T*k is small.
constexpr int kScanVecs = 8;  // 16-byte id loads in flight per lane in the pass over all ids

// Adds the valid ids of idx[i0, i1) to the LDS histogram h; returns this lane's count of invalid
// ids. 16-byte loads when the id array allows them, else 4-byte loads.
__device__ __forceinline__ int count_ids(const int32_t* __restrict__ idx, int i0, int i1, int E, int32_t* h) {
  int inval = 0;
  int head = i0;
  if ((reinterpret_cast<uintptr_t>(idx) & 15) == 0) {
    const int v0 = (i0 + 3) / 4, v1 = i1 / 4;  // whole 16-byte vectors inside [i0, i1)
    const int4* idx4 = reinterpret_cast<const int4*>(idx);
    for (int v = v0 + (int)threadIdx.x; v < v1; v += kLayoutThreads * kScanVecs) {
      int4 q[kScanVecs];
#pragma unroll
      for (int u = 0; u < kScanVecs; ++u) q[u] = idx4[min(v + u * kLayoutThreads, v1 - 1)];
#pragma unroll
      for (int u = 0; u < kScanVecs; ++u) {
        if (v + u * kLayoutThreads >= v1) break;
        const int e4[4] = {q[u].x, q[u].y, q[u].z, q[u].w};
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          if ((unsigned)e4[m] < (unsigned)E)
            atomicAdd(&h[e4[m]], 1);
          else
            ++inval;
        }
      }
    }
    if (v1 > v0) {  // the unaligned head and tail go through the 4-byte loop below
      for (int i = i0 + (int)threadIdx.x; i < 4 * v0; i += kLayoutThreads) {
        const int e = idx[i];
        if ((unsigned)e < (unsigned)E) atomicAdd(&h[e], 1); else ++inval;
      }
      head = 4 * v1;
    }
  }
  for (int i = head + (int)threadIdx.x; i < i1; i += kLayoutThreads) {
    const int e = idx[i];
    if ((unsigned)e < (unsigned)E) atomicAdd(&h[e], 1); else ++inval;
  }
  return inval;
}

__global__ void __launch_bounds__(kLayoutThreads)
    route_single_kernel(Geom G, const int32_t* __restrict__ idx, int32_t* __restrict__ send_cnt,
                        int32_t* __restrict__ rank_cnt, int32_t* __restrict__ expert_off, int32_t* __restrict__ rank_off,
                        int32_t* __restrict__ seg_off, int32_t* __restrict__ tok_nranks, int32_t* __restrict__ pair_row,
                        int32_t* __restrict__ pair_rslot, int32_t* __restrict__ recv_src, int32_t* __restrict__ recv_j,
                        int32_t* __restrict__ num_invalid) {
  extern __shared__ int32_t lds[];
  int32_t* h_pre = lds;                      // [E] pairs before the chunk, per expert
  int32_t* h_post = h_pre + G.E;             // [E] pairs from the chunk on, per expert
  int32_t* h_rank = h_post + G.E;            // [E] pairs of the source rank (its last chunk only)
  int32_t* base_r = h_rank + G.E;            // [R] first pairs of the rank's earlier tokens, per rank
  int32_t* own_r = base_r + G.R;             // [R] first pairs of this chunk's tokens, per rank
  int32_t* whe = own_r + G.R;                // [W][E]
  int32_t* whr = whe + kLayoutWaves * G.E;   // [W][R]
  int32_t* eoff = whr + kLayoutWaves * G.R;  // [E+1]
  int32_t* base_e = eoff + G.E + 1;          // [E]
  int32_t* ekey = base_e + G.E;              // [kMaxChunkPairs]
  int32_t* dkey = ekey + kMaxChunkPairs;     // [kMaxChunkPairs]
  int32_t* rs = dkey + kMaxChunkPairs;       // [kMaxChunkPairs]
  uint32_t* fm = reinterpret_cast<uint32_t*>(rs + kMaxChunkPairs);  // [kMaxChunkPairs]
  __shared__ int32_t red[kLayoutWaves];
  __shared__ int32_t scratch[kLayoutWaves];

  const int tid = threadIdx.x;
  const int b = blockIdx.x;
  const int s = b / G.NC;
  const int c = b - s * G.NC;
  const int t0 = c * G.CT;
  const int nt = max(0, min(G.CT, G.Tr - t0));
  const int np = nt * G.k;
  const int64_t g0 = (int64_t)s * G.Tr + t0;
  // T*k < 2^31 (checked on the host), so pair indices fit in int.
  const int npairs = (int)(G.T * G.k);
  const int rank_beg = s * G.Tr * G.k;
  const int chunk_beg = (int)(g0 * G.k);
  const int rank_end = rank_beg + G.Tr * G.k;
  const bool last = c == G.NC - 1;

  for (int i = tid; i < 3 * G.E + 2 * G.R + kLayoutWaves * (G.E + G.R); i += kLayoutThreads) lds[i] = 0;
  __syncthreads();

  int my_inval = count_ids(idx, 0, chunk_beg, G.E, h_pre);
  my_inval += count_ids(idx, chunk_beg, npairs, G.E, h_post);
  if (last) count_ids(idx, rank_beg, rank_end, G.E, h_rank);
  const int wsum = wave_sum(my_inval);
  if (lane_id() == 0) red[tid / kWave] = wsum;

  // This chunk's pairs (the loads hit in cache after the pass above).
  const int32_t* src = idx + chunk_beg;
  for (int i = tid; i < np; i += kLayoutThreads) {
    const int e = src[i];
    const bool ok = (unsigned)e < (unsigned)G.E;
    ekey[i] = ok ? e : -1;
    dkey[i] = ok ? small_div(e, G.inv_El) : -1;
  }

  // Dedup of the rank's earlier tokens [rank_beg/k, chunk_beg/k). With at most 64 ranks, one
  // thread per token keeps the ranks it has seen in a 64-bit mask; otherwise the earlier chunks
  // (all full) go through the rs buffer one at a time.
  if (G.R <= 64) {
    for (int t = tid; t < t0; t += kLayoutThreads) {
      const int32_t* it = idx + rank_beg + t * G.k;
      uint64_t seen = 0;
      for (int j = 0; j < G.k; ++j) {
        const int e = it[j];
        if ((unsigned)e >= (unsigned)G.E) continue;
        const int d = small_div(e, G.inv_El);
        if (!((seen >> d) & 1)) atomicAdd(&base_r[d], 1);
        seen |= 1ull << d;
      }
    }
    __syncthreads();
  } else {
    __syncthreads();
    for (int cc = 0; cc < c; ++cc) {
      const int npc = G.CT * G.k;
      const int32_t* srcc = idx + rank_beg + cc * npc;
      for (int i = tid; i < npc; i += kLayoutThreads) {
        const int e = srcc[i];
        rs[i] = (unsigned)e < (unsigned)G.E ? small_div(e, G.inv_El) : -1;
      }
      __syncthreads();
      for (int t = tid; t < G.CT; t += kLayoutThreads) {
        const int32_t* dt = rs + t * G.k;
        for (uint32_t m = first_rank_mask(dt, G.k); m; m &= m - 1) atomicAdd(&base_r[dt[__builtin_ctz(m)]], 1);
      }
      __syncthreads();
    }
  }
  for (int t = tid; t < nt; t += kLayoutThreads) {
    const int32_t* dt = dkey + t * G.k;
    const uint32_t mask = first_rank_mask(dt, G.k);
    for (uint32_t m = mask; m; m &= m - 1) atomicAdd(&own_r[dt[__builtin_ctz(m)]], 1);
    fm[t] = mask;
    tok_nranks[g0 + t] = __popc(mask);
  }

  // expert_off = exclusive scan of the expert totals; each thread owns a contiguous run of experts.
  {
    const int per = (G.E + kLayoutThreads - 1) / kLayoutThreads;
    const int e0 = min(G.E, tid * per), e1 = min(G.E, e0 + per);
    int sum = 0;
    for (int e = e0; e < e1; ++e) sum += h_pre[e] + h_post[e];
    int total;
    int run = block_exclusive_sum(sum, total, scratch);  // synchronises the workgroup
    for (int e = e0; e < e1; ++e) {
      eoff[e] = run;
      base_e[e] = run + h_pre[e];
      run += h_pre[e] + h_post[e];
    }
    if (tid == 0) eoff[G.E] = total;
  }
  __syncthreads();

  assign_chunk_rows(G, np, g0, eoff[G.E], ekey, dkey, fm, base_e, base_r, whe, whr, rs, pair_row, pair_rslot,
                    recv_src, recv_j);

  // Per-layout and per-rank outputs, each written by exactly one workgroup.
  if (b == 0) {
    for (int e = tid; e <= G.E; e += kLayoutThreads) expert_off[e] = eoff[e];
    for (int d = tid; d <= G.R; d += kLayoutThreads) rank_off[d] = eoff[d * G.El];
    if (tid == 0) {
      int n = 0;
      for (int w = 0; w < kLayoutWaves; ++w) n += red[w];
      num_invalid[0] = n;
    }
  }
  if (c == 0)  // the chunk starts the rank: h_pre counts the pairs of earlier ranks
    for (int e = tid; e < G.E; e += kLayoutThreads) seg_off[e * G.R + s] = eoff[e] + h_pre[e];
  if (last) {
    for (int e = tid; e < G.E; e += kLayoutThreads) send_cnt[s * G.E + e] = h_rank[e];
    for (int r = tid; r < G.R; r += kLayoutThreads) rank_cnt[s * G.R + r] = base_r[r] + own_r[r];
  }
}

// ------------------------------------------------------------------------------------ host
size_t single_lds_bytes(const Geom& g) {
  return sizeof(int32_t) * ((size_t)3 * g.E + 2 * g.R + (size_t)kLayoutWaves * (g.E + g.R) + (g.E + 1) + g.E +
                            4 * kMaxChunkPairs);
}

bool layout_single(const Geom& g) {
  return g.T * g.k <= kSingleMaxPairs && (int64_t)g.Tr * g.k <= kSingleMaxRankPairs &&
         single_lds_bytes(g) <= kSingleMaxLds;
}

static size_t finalize_lds_bytes(const Geom& g) {
  return sizeof(int32_t) * ((size_t)(g.E + 1) + g.E + g.R + (size_t)kLayoutWaves * (g.E + g.R) + 4 * kMaxChunkPairs);
}

hipError_t launch_layout(const Geom& g, const int32_t* idx, int32_t* ws, int32_t* send_cnt, int32_t* rank_cnt,
                         int32_t* expert_off, int32_t* rank_off, int32_t* seg_off, int32_t* tok_nranks,
                         int32_t* pair_row, int32_t* pair_rslot, int32_t* recv_src, int32_t* recv_j,
                         int32_t* num_invalid, hipStream_t stream) {
  if (layout_single(g)) {
    hipLaunchKernelGGL(route_single_kernel, dim3(g.nblk), dim3(kLayoutThreads), single_lds_bytes(g), stream, g, idx,
                       send_cnt, rank_cnt, expert_off, rank_off, seg_off, tok_nranks, pair_row, pair_rslot, recv_src,
                       recv_j, num_invalid);
    return hipGetLastError();
  }
  hipError_t err = launch_layout_counts(g, idx, ws, send_cnt, rank_cnt, tok_nranks, num_invalid, stream);
  if (err != hipSuccess) return err;
  return launch_layout_finalize(g, idx, ws, expert_off, rank_off, seg_off, pair_row, pair_rslot, recv_src, recv_j,
                                stream);
}

hipError_t launch_layout_finalize(const Geom& g, const int32_t* idx, int32_t* ws, int32_t* expert_off,
                                  int32_t* rank_off, int32_t* seg_off, int32_t* pair_row, int32_t* pair_rslot,
                                  int32_t* recv_src, int32_t* recv_j, hipStream_t stream) {
  const WsLayout wl = ws_layout(g);
  hipLaunchKernelGGL(route_finalize_kernel, dim3(g.nblk), dim3(kLayoutThreads), finalize_lds_bytes(g), stream, g,
                     idx, ws + wl.chunk_e, ws + wl.chunk_r, ws + wl.recv_cnt, ws + wl.seg_rel,
                     reinterpret_cast<const uint32_t*>(ws + wl.fmask), expert_off, rank_off, seg_off, pair_row,
                     pair_rslot, recv_src, recv_j);
  return hipGetLastError();
}

hipError_t launch_layout_counts(const Geom& g, const int32_t* idx, int32_t* ws, int32_t* send_cnt, int32_t* rank_cnt,
                                int32_t* tok_nranks, int32_t* num_invalid, hipStream_t stream) {
  const WsLayout wl = ws_layout(g);
  int32_t* chunk_e = ws + wl.chunk_e;
  int32_t* chunk_r = ws + wl.chunk_r;
  int32_t* recv_cnt = ws + wl.recv_cnt;
  int32_t* inval = ws + wl.inval;
  int32_t* seg_rel = ws + wl.seg_rel;
  uint32_t* fmask = reinterpret_cast<uint32_t*>(ws + wl.fmask);

  const size_t lds1 = sizeof(int32_t) * ((size_t)g.E + g.R + kMaxChunkPairs);
  hipLaunchKernelGGL(route_hist_kernel, dim3(g.nblk), dim3(kLayoutThreads), lds1, stream, g, idx, tok_nranks,
                     chunk_e, chunk_r, inval, fmask);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;

  hipLaunchKernelGGL(route_scan_kernel, dim3(g.E + g.R + 1), dim3(kLayoutThreads), 0, stream, g, chunk_e, chunk_r,
                     inval, recv_cnt, send_cnt, rank_cnt, seg_rel, num_invalid);
  return hipGetLastError();
}

}  // namespace epl
