// MoE dispatch on one GPU: write each token's row into the packed receive row of every valid
// (token, expert) pair.
//
// This is the paper's Token-Sending into pre-partitioned receive space (Implementation, global
// load/store; Background phase 2). Token-Reordering is fused in: the layout has already fixed
// every row, so each copy lands in its final slot.
//
// Work is cut into equal units, each a (token, column chunk) pair, one unit per wave. Every unit
// moves at most k copies of the same number of bytes, so the units are as balanced as the
// paper's equal token slices (Hierarchical Token-level Scheduling). Fine units also keep the
// last partial round of waves short. The token's chunk is read once with 16-byte loads and
// written k times with 16-byte stores.
//
// The fp8 variant quantises while copying. For each 128-element block the scale is
// s = max|x| / 448, and each element is stored as q = E4M3(x / s), RNE and saturating. It
// writes the same q row and scale row to all k destinations.
#include "rows_body.h"

namespace epl {

// Waves per SIMD of the plain bf16 kernel. The instance that reads a large x through buffer loads
// is held at exactly 6; the other is left unconstrained (1 to 8, which compiles to the same code
// as no attribute; its register use allows 8). Layout -> dispatch -> combine with the input
// rotated, dispatch per call, two runs each, caps 3 / 4 / 6 / unconstrained:
// * EP=32 prefill (buffer loads): 3278-3281 / 3242 / 3238-3242 / 3279-3280 us;
// * EP=256 (buffer loads): 385.9-386.5 / 382.2-382.5 / 375.9-376.7 / 380.8-381.0 us;
// * EP=64 decode (plain loads): 180.9-181.1 / 181.5 / 179.7-179.8 / 176.2-176.6 us.
constexpr int bf16_min_waves(bool buf_x) { return buf_x ? 6 : 1; }
constexpr int bf16_max_waves(bool buf_x) { return buf_x ? 6 : 8; }
template <bool BUF_X>
__global__ void __launch_bounds__(kPlainThreads)
    __attribute__((amdgpu_waves_per_eu(bf16_min_waves(BUF_X), bf16_max_waves(BUF_X))))
    dispatch_bf16_kernel(const u32x4* __restrict__ x, const int32_t* __restrict__ pair_row, u32x4* __restrict__ recv,
                         int64_t T, int k, int nv, int pv, int chunks, int64_t cap) {
  const int lane = threadIdx.x % kWave;
  const int64_t units = T * chunks;
  const int64_t stride = (int64_t)gridDim.x * kPlainWaves;
  for (int64_t u = (int64_t)blockIdx.x * kPlainWaves + threadIdx.x / kWave; u < units; u += stride) {
    const int64_t g = u / chunks;
    dispatch_bf16_unit<BUF_X>(
        x, [&] { return lane < k ? pair_row[g * k + lane] : -1; }, recv, g, (int)(u - g * chunks), k, nv, pv, cap,
        lane);
  }
}

// The fp8 kernel is capped at kFp8WavesPerSimd waves per SIMD. The compiler enforces the cap by
// reserving a larger register budget. Each wave writes up to k scattered 1 KiB q rows per 2 KiB of
// input, so fewer resident waves keep fewer concurrent random writes in flight; too few leave the
// per-element IEEE divisions of the quantiser exposed. Skewed fp8 EP=64, layout -> dispatch ->
// combine with the input rotated, dispatch per call over three alternating runs each:
// * 2 waves: 239.2-239.6 us;
// * 3 waves: 209.2-209.7 us;
// * 4 waves: 220.7-221.3 us;
// * 6 waves: 222.6-223.4 us;
// * 8 waves (uncapped): 222.6-222.8 us.
// With 2 waves, multiplying by a reciprocal instead of dividing (not the defined rounding) also
// brought it to 221 us, which places the 2-wave loss in the division latency.
constexpr int kFp8WavesPerSimd = 3;
__global__ void __launch_bounds__(kFp8Threads) __attribute__((amdgpu_waves_per_eu(kFp8WavesPerSimd, kFp8WavesPerSimd)))
    dispatch_fp8_kernel(const u32x4* __restrict__ x, const int32_t* __restrict__ pair_row, u32x4* __restrict__ recv,
                        float* __restrict__ recv_scale, int64_t T, int k, int H, int pq, int npass, int64_t cap) {
  const int lane = threadIdx.x % kWave;
  const int64_t units = T * npass;
  const int64_t stride = (int64_t)gridDim.x * kFp8Waves;
  for (int64_t u = (int64_t)blockIdx.x * kFp8Waves + threadIdx.x / kWave; u < units; u += stride) {
    const int64_t g = u / npass;
    dispatch_fp8_unit(x, [&] { return lane < k ? pair_row[g * k + lane] : -1; }, recv, recv_scale, g,
                      (int)(u - g * npass), k, H, pq, cap, lane);
  }
}

hipError_t launch_dispatch_bf16(const void* x, const int32_t* pair_row, void* recv, int64_t T, int k, int H,
                                int pitch, int64_t cap, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  const int nv = H / 8;
  const int chunks = (nv + kBf16Cols - 1) / kBf16Cols;
  const int64_t units = T * chunks;
  const dim3 grid((unsigned)std::min<int64_t>((units + kPlainWaves - 1) / kPlainWaves, 1 << 30));
  if (T * (int64_t)H * 2 >= kBufferLoadXBytes)
    hipLaunchKernelGGL(dispatch_bf16_kernel<true>, grid, dim3(kPlainThreads), 0, stream,
                       static_cast<const u32x4*>(x), pair_row, static_cast<u32x4*>(recv), T, k, nv, pitch / 8, chunks,
                       cap);
  else
    hipLaunchKernelGGL(dispatch_bf16_kernel<false>, grid, dim3(kPlainThreads), 0, stream,
                       static_cast<const u32x4*>(x), pair_row, static_cast<u32x4*>(recv), T, k, nv, pitch / 8, chunks,
                       cap);
  return hipGetLastError();
}

hipError_t launch_dispatch_fp8(const void* x, const int32_t* pair_row, void* recv, float* recv_scale, int64_t T,
                               int k, int H, int pitch, int64_t cap, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  const int npass = (H + 1023) / 1024;
  const int64_t units = T * npass;
  const dim3 grid((unsigned)std::min<int64_t>((units + kFp8Waves - 1) / kFp8Waves, 1 << 30));
  hipLaunchKernelGGL(dispatch_fp8_kernel, grid, dim3(kFp8Threads), 0, stream, static_cast<const u32x4*>(x),
                     pair_row, static_cast<u32x4*>(recv), recv_scale, T, k, H, pitch / 16, npass, cap);
  return hipGetLastError();
}

// ------------------------------------------------------------------------ layout finalize fused into dispatch
// epl_layout_dispatch runs K1 and K2 of the layout, then one kernel that does both the layout's
// finalize step and the dispatch. No workgroup waits on another; the rows of each token are worked
// out inside its workgroup from what K1 and K2 left in the workspace, with exactly the definitions
// route_finalize_kernel applies to a whole chunk:
// * row of pair (g, j) = first row of its expert (exclusive prefix of recv_cnt)
//                      + rows of the expert before the token's chunk (K2's chunk offsets)
//                      + earlier pairs of the chunk with the same expert (an LDS histogram of the
//                        chunk's earlier tokens plus a ballot match over the token's own choices);
// * slot of a first pair = slots of its rank before the chunk (K2) + earlier first pairs of the
//   chunk bound for that rank; other valid pairs share the slot of their token's first pair on
//   the same rank.
// A workgroup's waves cover consecutive units, so they share few tokens (one when a row has as
// many column chunks as the workgroup has waves). Wave w computes the rows of the workgroup's
// w-th token, writes that token's pair_row, pair_rslot, recv_src and recv_j, and leaves the rows
// in LDS for the other waves. A few extra workgroups at the start of the grid write expert_off,
// rank_off and seg_off. The loads of x are issued before the row computation, so they are in
// flight while it runs.
template <bool BUF_X>
__global__ void __launch_bounds__(kDispatchThreads)
    fused_bf16_kernel(FusedLayout F, const u32x4* __restrict__ x, u32x4* __restrict__ recv, int nv, int pv,
                      int chunks, int64_t cap, int unit_grid, int nmeta) {
  extern __shared__ int32_t lds[];
  // The metadata workgroups come first in the grid, so that they run alongside the units
  // instead of after them.
  if ((int)blockIdx.x < nmeta) {
    fused_meta_block<false>(F, (int)blockIdx.x, nmeta, lds);
    return;
  }
  const int blk = (int)blockIdx.x - nmeta;
  const int lane = threadIdx.x % kWave;
  const int w = threadIdx.x / kWave;
  const int k = F.G.k;
  int32_t* rows_lds = lds;  // [kWavesPerBlock][k]
  int32_t* hist = lds + kWavesPerBlock * EPL_MAX_TOPK + w * (F.G.E + F.G.R);
  const int64_t units = F.G.T * chunks;
  const int64_t stride = (int64_t)unit_grid * kWavesPerBlock;
  // The loop bound depends on the workgroup's first unit only, so every wave runs the same
  // iterations and reaches the same barriers.
  for (int64_t ub = (int64_t)blk * kWavesPerBlock; ub < units; ub += stride) {
    const int64_t g_first = ub / chunks;
    const int64_t g_last = std::min(units - 1, ub + kWavesPerBlock - 1) / chunks;
    const int64_t u = ub + w;
    const bool active = u < units;
    const int64_t g = (active ? u : units - 1) / chunks;
    const int c = (int)((active ? u : units - 1) - g * chunks);
    dispatch_bf16_unit<BUF_X>(
        x,
        [&] {
          if (w <= g_last - g_first) {
            const int r = token_rows<false>(F, g_first + w, true, hist, lane);
            if (lane < k) rows_lds[w * k + lane] = r;
          }
          __syncthreads();
          const int r = lane < k ? rows_lds[(g - g_first) * k + lane] : -1;
          __syncthreads();  // every wave has its rows before the next iteration rewrites them
          return r;
        },
        recv, g, c, k, nv, pv, cap, lane, active);
  }
}

bool fused_dispatch_ok(const Geom& g, bool fp8) {
  return !fp8 && g.CT * g.k <= kFusedSlots * kWave && g.E <= kFusedPer * kWave;
}

hipError_t launch_fused_dispatch(const Geom& g, const int32_t* idx, int32_t* ws, int32_t* expert_off,
                                 int32_t* rank_off, int32_t* seg_off, int32_t* pair_row, int32_t* pair_rslot,
                                 int32_t* recv_src, int32_t* recv_j, const void* x, void* recv, int H, int pitch,
                                 int64_t cap, hipStream_t stream) {
  const WsLayout wl = ws_layout(g);
  const FusedLayout F{g,          idx,          ws + wl.chunk_e, ws + wl.chunk_r,
                      ws + wl.recv_cnt, ws + wl.seg_rel, reinterpret_cast<const uint32_t*>(ws + wl.fmask),
                      expert_off, rank_off,     seg_off,         pair_row,
                      pair_rslot, recv_src,     recv_j};
  const int nmeta = (int)std::max<int64_t>(1, ((int64_t)g.E * g.R + 4 * kDispatchThreads - 1) / (4 * kDispatchThreads));
  const int chunks = (H / 8 + kBf16Cols - 1) / kBf16Cols;
  const int64_t units = g.T * chunks;
  const int unit_grid = (int)std::min<int64_t>((units + kWavesPerBlock - 1) / kWavesPerBlock, 1 << 30);
  const dim3 grid((unsigned)(unit_grid + nmeta));
  const size_t lds = sizeof(int32_t) * std::max<size_t>((size_t)kWavesPerBlock * (EPL_MAX_TOPK + g.E + g.R),
                                                        (size_t)g.E + 1);
  const bool buf_x = g.T * (int64_t)H * 2 >= kBufferLoadXBytes;
  const u32x4* xv = static_cast<const u32x4*>(x);
  u32x4* rv = static_cast<u32x4*>(recv);
  if (buf_x)
    hipLaunchKernelGGL(fused_bf16_kernel<true>, grid, dim3(kDispatchThreads), lds, stream, F, xv, rv, H / 8,
                       pitch / 8, chunks, cap, unit_grid, nmeta);
  else
    hipLaunchKernelGGL(fused_bf16_kernel<false>, grid, dim3(kDispatchThreads), lds, stream, F, xv, rv, H / 8,
                       pitch / 8, chunks, cap, unit_grid, nmeta);
  return hipGetLastError();
}

// ------------------------------------------------------------------------ diagnostics
__global__ void debug_e4m3_kernel(const float* __restrict__ in, uint8_t* __restrict__ out, int64_t n) {
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= n) return;
  float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int t = 0; t < 4 && i + t < n; ++t) v[t] = in[i + t];
  const uint32_t q = f32x4_to_e4m3x4(v[0], v[1], v[2], v[3]);
  for (int t = 0; t < 4 && i + t < n; ++t) out[i + t] = (uint8_t)(q >> (8 * t));
}

hipError_t launch_debug_e4m3(const float* in, uint8_t* out, int64_t n, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  const int64_t threads = (n + 3) / 4;
  hipLaunchKernelGGL(debug_e4m3_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, stream, in, out, n);
  return hipGetLastError();
}

}  // namespace epl
