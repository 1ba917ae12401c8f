// Hierarchical token-level scheduling (Hierarchical Token-level Scheduling: Latency
// Homogenization and the Hardware-Accelerated Mapper).
//
// The paper cuts the pairs one source sends into n equal contiguous slices, one per worker
// (Token-level Load Partition), after reordering the experts so that every slice holds a similar
// mix of hop classes (Expert Remapping via Logical Matrix Transposition): the experts are laid row
// by row into a virtual matrix with one row per worker and read back column by column. A worker
// finds where its slice starts with Algorithm 1 over the cumulative counts of the remapped
// sequence. The per-hop capacity bound v_{j,h} <= ceil(V_h / n) is what the remap aims for.
//
// Two kernels:
// * hop_schedule_kernel, one workgroup per source rank: the remapped sequence and its cumulative
//   counts in LDS (also one cumulative count per hop class), then for every worker the slice's
//   first expert and offset (Algorithm 1's lookup) and its pairs per hop class;
// * dispatch_scheduled_kernel, one workgroup per (source rank, worker): the worker's slice of
//   pairs, taken in the remapped order, each copied from its token's row of x into its packed
//   receive row (quantised to fp8 on the way for fp8 payloads). The rows are those of the layout, so
//   the output equals epl_dispatch's; only the order of the writes and the split of the work across
//   workgroups follow the schedule. Each pair reads its token's row again, as the paper's per-pair
//   sends do (k reads of a token instead of one).
#include "layout_body.h"
#include "rows_body.h"

namespace epl {

constexpr int kScheduleThreads = kLayoutThreads;  // block_exclusive_sum works on 256-thread blocks
constexpr int kSchedulePer = EPL_MAX_EXPERTS / kScheduleThreads;  // remapped positions per thread

// Position of expert e in the remapped sequence of a matrix with `rows` rows: c = ceil(E / rows)
// columns, expert e in row e / c and column e % c, read column by column skipping the empty
// cells. The first full = E / c rows hold c experts each and the next row holds the other
// rem = E - full * c, so column col holds full + (col < rem) experts.
__device__ __forceinline__ int remap_position(int e, int E, int rows) {
  const int c = (E + rows - 1) / rows;
  const int full = E / c;
  const int rem = E - full * c;
  const int row = e / c, col = e - row * c;
  return col * full + min(col, rem) + row;
}

// A source rank's pairs in the remapped expert sequence: exp_at[i] is the i-th expert (-1 for an
// order entry outside [0, E), which counts as an expert without pairs), cnt_at[i] its pair count,
// cum[0..E] the exclusive prefix sums (cum[E] = the rank's pairs). With order == nullptr the
// sequence is the transposition with `rows` rows. Every thread of the block calls it.
__device__ __forceinline__ void remapped_counts(const int32_t* __restrict__ send_row, const int32_t* __restrict__ order,
                                                int E, int rows, int32_t* exp_at, int32_t* cnt_at, int32_t* cum,
                                                int* scratch) {
  for (int i = threadIdx.x; i < E; i += kScheduleThreads) {
    if (order) {
      const int e = order[i];
      const bool ok = e >= 0 && e < E;
      exp_at[i] = ok ? e : -1;
      cnt_at[i] = ok ? send_row[e] : 0;
    } else {
      const int p = remap_position(i, E, rows);
      exp_at[p] = i;
      cnt_at[p] = send_row[i];
    }
  }
  __syncthreads();
  int v[kSchedulePer];
  int sum = 0;
#pragma unroll
  for (int q = 0; q < kSchedulePer; ++q) {
    const int i = threadIdx.x * kSchedulePer + q;
    v[q] = i < E ? cnt_at[i] : 0;
    sum += v[q];
  }
  int total;
  int pre = block_exclusive_sum(sum, total, scratch);
#pragma unroll
  for (int q = 0; q < kSchedulePer; ++q) {
    const int i = threadIdx.x * kSchedulePer + q;
    if (i < E) cum[i] = pre;
    pre += v[q];
  }
  if (threadIdx.x == 0) cum[E] = total;
  __syncthreads();
}

// One workgroup per source rank s. Worker j's slice is positions [j*m/n, (j+1)*m/n) of the rank's
// m pairs in the remapped sequence. Pairs per hop class come from per-class cumulative counts:
// F_h(t), the class-h pairs among the first t positions, is cumh[h][i] plus t - cum[i] when the
// expert at index i (the one holding position t) is of class h; a slice holds F_h(hi) - F_h(lo).
__global__ void __launch_bounds__(kScheduleThreads)
    hop_schedule_kernel(const int32_t* __restrict__ send_cnt, const int32_t* __restrict__ order,
                        const int32_t* __restrict__ hop, int R, int E, int rows, int n, int NH,
                        int32_t* __restrict__ start_expert, int32_t* __restrict__ start_offset,
                        int32_t* __restrict__ class_cnt) {
  __shared__ int32_t exp_at[EPL_MAX_EXPERTS];
  __shared__ int32_t cnt_at[EPL_MAX_EXPERTS];
  __shared__ int32_t cls_at[EPL_MAX_EXPERTS];
  __shared__ int32_t cum[EPL_MAX_EXPERTS + 1];
  __shared__ int32_t cumh[EPL_MAX_HOP_CLASSES][EPL_MAX_EXPERTS + 1];
  __shared__ int scratch[kLayoutWaves];
  const int s = blockIdx.x;
  const int El = E / R;
  remapped_counts(send_cnt + (int64_t)s * E, order, E, rows, exp_at, cnt_at, cum, scratch);
  for (int i = threadIdx.x; i < E; i += kScheduleThreads) {
    const int e = exp_at[i];
    cls_at[i] = e >= 0 ? hop[(int64_t)s * R + e / El] : -1;
  }
  __syncthreads();
  for (int h = 0; h < NH; ++h) {
    int v[kSchedulePer];
    int sum = 0;
#pragma unroll
    for (int q = 0; q < kSchedulePer; ++q) {
      const int i = threadIdx.x * kSchedulePer + q;
      v[q] = (i < E && cls_at[i] == h) ? cnt_at[i] : 0;
      sum += v[q];
    }
    int total;
    int pre = block_exclusive_sum(sum, total, scratch);
#pragma unroll
    for (int q = 0; q < kSchedulePer; ++q) {
      const int i = threadIdx.x * kSchedulePer + q;
      if (i < E) cumh[h][i] = pre;
      pre += v[q];
    }
    if (threadIdx.x == 0) cumh[h][E] = total;
  }
  __syncthreads();
  const int64_t m = cum[E];
  for (int j = threadIdx.x; j < n; j += kScheduleThreads) {
    const int64_t lo = (int64_t)j * m / n, hi = (int64_t)(j + 1) * m / n;
    const int64_t w = (int64_t)s * n + j;
    int32_t* cnt = class_cnt + w * NH;
    if (hi <= lo) {
      start_expert[w] = -1;
      start_offset[w] = -1;
      for (int h = 0; h < NH; ++h) cnt[h] = 0;
      continue;
    }
    const int ilo = quaternary_find(cum, E, lo);
    start_expert[w] = exp_at[ilo];
    start_offset[w] = (int32_t)(lo - cum[ilo]);
    const int ihi = hi < m ? quaternary_find(cum, E, hi) : E;
    for (int h = 0; h < NH; ++h) {
      const int64_t f_lo = cumh[h][ilo] + (cls_at[ilo] == h ? lo - cum[ilo] : 0);
      const int64_t f_hi = ihi < E ? cumh[h][ihi] + (cls_at[ihi] == h ? hi - cum[ihi] : 0) : cumh[h][E];
      cnt[h] = (int32_t)(f_hi - f_lo);
    }
  }
}

// One workgroup per (source rank s, worker j). The slice's positions are handled in
// batches of one per thread: each thread locates its position (Algorithm 1's lookup over the
// remapped cumulative counts), takes the pair's packed row seg_off[e][s] + offset and its token
// recv_src[row], and shares both through LDS; the waves then copy the batch's rows, one
// (row, 4 KiB column chunk) unit per wave as the token-major dispatch does, with one destination.
// FP8: each row is quantised as it is copied, by the fp8 dispatch's unit (token, 1024-element pass)
// with one destination; units per row is then the number of passes.
template <bool BUF_X, bool FP8>
__global__ void __launch_bounds__(kScheduleThreads)
    dispatch_scheduled_kernel(const u32x4* __restrict__ x, const int32_t* __restrict__ send_cnt,
                              const int32_t* __restrict__ seg_off, const int32_t* __restrict__ recv_src,
                              u32x4* __restrict__ recv, float* __restrict__ recv_scale, int R, int E, int rows, int n,
                              int64_t T, int k, int H, int pitch, int chunks, int64_t cap) {
  __shared__ int32_t exp_at[EPL_MAX_EXPERTS];
  __shared__ int32_t cnt_at[EPL_MAX_EXPERTS];
  __shared__ int32_t cum[EPL_MAX_EXPERTS + 1];
  __shared__ int32_t row_lds[kScheduleThreads];
  __shared__ int32_t src_lds[kScheduleThreads];
  __shared__ int scratch[kLayoutWaves];
  // Workgroup i runs on XCD i % 8; xcd_chunk gives each XCD a contiguous range of (source, worker)
  // slices, so a source's workers share one L2 for the token rows they all read.
  const int slice = xcd_chunk((int)blockIdx.x, (int)gridDim.x);
  const int s = slice / n;
  const int j = slice - s * n;
  const int lane = threadIdx.x % kWave;
  const int64_t Tk = T * k;
  remapped_counts(send_cnt + (int64_t)s * E, nullptr, E, rows, exp_at, cnt_at, cum, scratch);
  const int64_t m = cum[E];
  const int64_t lo = (int64_t)j * m / n, hi = (int64_t)(j + 1) * m / n;
  for (int64_t base = lo; base < hi; base += kScheduleThreads) {
    const int nb = (int)std::min<int64_t>(kScheduleThreads, hi - base);
    if (threadIdx.x < nb) {
      const int64_t p = base + threadIdx.x;
      const int i = quaternary_find(cum, E, p);
      const int e = exp_at[i];
      const int row = seg_off[(int64_t)e * R + s] + (int)(p - cum[i]);
      const bool ok = row >= 0 && row < Tk;
      row_lds[threadIdx.x] = ok ? row : -1;
      src_lds[threadIdx.x] = ok ? recv_src[row] : -1;
    }
    __syncthreads();
    const int units = nb * chunks;
    for (int u = threadIdx.x / kWave; u < units; u += kScheduleThreads / kWave) {
      const int q = u / chunks;
      const int row = row_lds[q];
      const int g = src_lds[q];
      if (g < 0 || g >= T) continue;  // only a layout that does not belong to x gets here
      if constexpr (FP8)
        dispatch_fp8_unit(x, [&] { return row; }, recv, recv_scale, g, u - q * chunks, 1, H, pitch / 16, cap, lane);
      else
        dispatch_bf16_unit<BUF_X>(x, [&] { return row; }, recv, g, u - q * chunks, 1, H / 8, pitch / 8, cap, lane);
    }
    __syncthreads();  // the batch's rows are consumed before the next batch overwrites them
  }
}

hipError_t launch_hop_schedule(const int32_t* send_cnt, const int32_t* order, const int32_t* hop, int R, int E,
                               int rows, int n, int NH, int32_t* start_expert, int32_t* start_offset,
                               int32_t* class_cnt, hipStream_t stream) {
  hipLaunchKernelGGL(hop_schedule_kernel, dim3((unsigned)R), dim3(kScheduleThreads), 0, stream, send_cnt, order, hop,
                     R, E, rows, n, NH, start_expert, start_offset, class_cnt);
  return hipGetLastError();
}

hipError_t launch_dispatch_scheduled(const void* x, const int32_t* send_cnt, const int32_t* seg_off,
                                     const int32_t* recv_src, void* recv, float* recv_scale, int R, int E, int rows,
                                     int n, int64_t T, int k, int H, int pitch, int64_t cap, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  const bool fp8 = recv_scale != nullptr;
  const int chunks = fp8 ? (H + 1023) / 1024 : (H / 8 + kBf16Cols - 1) / kBf16Cols;
  const dim3 grid((unsigned)((int64_t)R * n));
  const u32x4* xv = static_cast<const u32x4*>(x);
  u32x4* rv = static_cast<u32x4*>(recv);
  if (fp8)
    hipLaunchKernelGGL((dispatch_scheduled_kernel<false, true>), grid, dim3(kScheduleThreads), 0, stream, xv, send_cnt,
                       seg_off, recv_src, rv, recv_scale, R, E, rows, n, T, k, H, pitch, chunks, cap);
  else if (T * (int64_t)H * 2 >= kBufferLoadXBytes)
    hipLaunchKernelGGL((dispatch_scheduled_kernel<true, false>), grid, dim3(kScheduleThreads), 0, stream, xv, send_cnt,
                       seg_off, recv_src, rv, nullptr, R, E, rows, n, T, k, H, pitch, chunks, cap);
  else
    hipLaunchKernelGGL((dispatch_scheduled_kernel<false, false>), grid, dim3(kScheduleThreads), 0, stream, xv,
                       send_cnt, seg_off, recv_src, rv, nullptr, R, E, rows, n, T, k, H, pitch, chunks, cap);
  return hipGetLastError();
}

}  // namespace epl
