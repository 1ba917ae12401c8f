// MoE combine on one GPU: gate-weighted gather-reduce of expert output rows back into token order
// (the paper's combine: gather expert outputs and restore the original token order).
//
// One wave per token. The workgroup stages its tokens' k packed-row indices and k gate weights
// in LDS with one coalesced load; each wave reads its own token's entries from there. The wave
// then walks the row in passes of VPL 16-byte vectors per lane. Per pass it issues the loads of
// up to KG expert rows before consuming any (many gathers in flight), then folds them in the
// token's own j order, acc = fmaf(w_j, y_j, acc), in fp32 starting from +0. Results are rounded
// to bf16 (RNE) and stored as 16-byte vectors. Pairs with row < 0 (invalid expert id) are
// skipped.
#include "epl_internal.h"

namespace epl {

constexpr int kCombineThreads = 256;
constexpr int kCombineTokens = kCombineThreads / kWave;

template <int KG, int VPL>
__global__ void __launch_bounds__(kCombineThreads)
    combine_kernel(const u32x4* __restrict__ y, const float* __restrict__ w, const int32_t* __restrict__ pair_row,
                   u32x4* __restrict__ out, int64_t T, int k, int nv) {
  __shared__ int32_t rows_lds[kCombineTokens * EPL_MAX_TOPK];
  __shared__ float w_lds[kCombineTokens * EPL_MAX_TOPK];
  const int64_t g_first = (int64_t)blockIdx.x * kCombineTokens;
  const int ntok = (int)min<int64_t>(kCombineTokens, T - g_first);
  for (int i = threadIdx.x; i < ntok * k; i += kCombineThreads) {
    rows_lds[i] = pair_row[g_first * k + i];
    w_lds[i] = w[g_first * k + i];
  }
  __syncthreads();

  const int lane = threadIdx.x % kWave;
  const int wv = threadIdx.x / kWave;
  if (wv >= ntok) return;
  const int64_t g = g_first + wv;
  const int32_t* rows = rows_lds + wv * k;
  const float* ws = w_lds + wv * k;

  for (int v0 = 0; v0 < nv; v0 += kWave * VPL) {
    float acc[VPL][8];
#pragma unroll
    for (int u = 0; u < VPL; ++u)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[u][e] = 0.0f;

    for (int j0 = 0; j0 < k; j0 += KG) {
      u32x4 buf[KG][VPL];
#pragma unroll
      for (int jj = 0; jj < KG; ++jj) {
        const int j = j0 + jj;
        const int row = (j < k) ? rows[j] : -1;
        if (row < 0) continue;
        const u32x4* src = y + (int64_t)row * nv;
#pragma unroll
        for (int u = 0; u < VPL; ++u) {
          const int v = v0 + u * kWave + lane;
          if (v < nv) buf[jj][u] = __builtin_nontemporal_load(src + v);
        }
      }
#pragma unroll
      for (int jj = 0; jj < KG; ++jj) {
        const int j = j0 + jj;
        if (j >= k) break;
        const int row = rows[j];
        if (row < 0) continue;
        const float wj = ws[j];
#pragma unroll
        for (int u = 0; u < VPL; ++u) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            acc[u][2 * i] = fmaf(wj, bf16lo_to_f32(buf[jj][u][i]), acc[u][2 * i]);
            acc[u][2 * i + 1] = fmaf(wj, bf16hi_to_f32(buf[jj][u][i]), acc[u][2 * i + 1]);
          }
        }
      }
    }
#pragma unroll
    for (int u = 0; u < VPL; ++u) {
      const int v = v0 + u * kWave + lane;
      if (v < nv) {
        u32x4 o;
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = f32x2_to_bf16x2(acc[u][2 * i], acc[u][2 * i + 1]);
        out[g * nv + v] = o;
      }
    }
  }
}

hipError_t launch_combine(const void* y, const float* w, const int32_t* pair_row, void* out, int64_t T, int k,
                          int H, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  const int nv = H / 8;
  const dim3 grid((unsigned)((T + kCombineTokens - 1) / kCombineTokens));
  const u32x4* yv = static_cast<const u32x4*>(y);
  u32x4* ov = static_cast<u32x4*>(out);
  hipLaunchKernelGGL((combine_kernel<8, 2>), grid, dim3(kCombineThreads), 0, stream, yv, w, pair_row, ov, T, k, nv);
  return hipGetLastError();
}

// ------------------------------------------------------------------------ diagnostics
__global__ void debug_bf16_kernel(const float* __restrict__ in, uint16_t* __restrict__ out, int64_t n) {
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 2;
  if (i >= n) return;
  const float a = in[i];
  const float b = (i + 1 < n) ? in[i + 1] : 0.0f;
  const uint32_t p = f32x2_to_bf16x2(a, b);
  out[i] = (uint16_t)(p & 0xFFFFu);
  if (i + 1 < n) out[i + 1] = (uint16_t)(p >> 16);
}

hipError_t launch_debug_bf16(const float* in, uint16_t* out, int64_t n, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  const int64_t threads = (n + 1) / 2;
  hipLaunchKernelGGL(debug_bf16_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, stream, in, out, n);
  return hipGetLastError();
}

}  // namespace epl
