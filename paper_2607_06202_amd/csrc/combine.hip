// MoE combine on one GPU: gate-weighted gather-reduce of expert output rows back into token order
// (the paper's combine: gather expert outputs and restore the original token order).
//
// Work is cut into equal units, each a (token, column chunk) pair, one unit per wave. The
// workgroup stages its tokens' k packed-row indices and k gate weights in LDS with one coalesced
// load. A wave issues the 16-byte loads of up to 8 expert rows before consuming any (many
// gathers in flight). It then folds them in the token's own j order, acc = fmaf(w_j, y_j, acc),
// in fp32 starting from +0, rounds to bf16 (RNE) and stores 16-byte vectors with sc1+nt stores
// (plain stores leave dirty lines whose write-back the next kernel pays for). Pairs with
// row < 0 (invalid expert id) are skipped.
#include "epl_internal.h"

namespace epl {

// Two waves per workgroup. Whole layer, two runs each, combine us with 128 / 256 / 512 threads:
// decode 190.8-190.9 / 191.5-191.8 / 191.7-192.1; prefill 2875-2877 / 2897 / 2868;
// skewed fp8 341.5-341.8 / 341.0 / 350; EP=256 365.8 / 366.0-367.2 / 363.2-363.4.
constexpr int kCombineThreads = 128;
constexpr int kCombineWaves = kCombineThreads / kWave;
constexpr int kGather = 8;                           // expert rows loaded before any is consumed
// Column chunk of a unit: VPL 16-byte vectors per lane, so 1 KiB (VPL = 1) or 2 KiB (VPL = 2) of each
// of the token's rows.
template <int VPL>
constexpr int combine_cols() { return kWave * VPL; }

// One unit: gather chunk c of the token's k expert rows and fold them in j order. Row
// indices and weights are wave-uniform and are read into scalar registers, so skipping an
// invalid pair is a scalar branch. With k <= kGather all loads are issued before the first
// fmaf. Larger k walks the choices in groups of kGather, still in j order.
template <bool SMALL_K, int VPL>
__device__ __forceinline__ void combine_unit(const u32x4* __restrict__ y, const int32_t* rows, const float* ws,
                                             u32x4* __restrict__ out, int64_t g, int c, int k, int nv, int pv,
                                             int lane) {
  int v[VPL], vl[VPL];
#pragma unroll
  for (int q = 0; q < VPL; ++q) {
    v[q] = c * combine_cols<VPL>() + q * kWave + lane;
    vl[q] = min(v[q], nv - 1);  // clamped so the gather loads need no per-lane branch
  }
  float acc[VPL][8];
#pragma unroll
  for (int q = 0; q < VPL; ++q)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[q][e] = 0.0f;
  const int kend = SMALL_K ? kGather : k;
  for (int j0 = 0; j0 < kend; j0 += kGather) {
    u32x4 buf[kGather][VPL];
#pragma unroll
    for (int jj = 0; jj < kGather; ++jj) {
      const int j = j0 + jj;
      const int row = j < k ? __builtin_amdgcn_readfirstlane(rows[j]) : -1;
      if (row >= 0) {
#pragma unroll
        for (int q = 0; q < VPL; ++q) buf[jj][q] = __builtin_nontemporal_load(y + (int64_t)row * pv + vl[q]);
      }
    }
#pragma unroll
    for (int jj = 0; jj < kGather; ++jj) {
      const int j = j0 + jj;
      const int row = j < k ? __builtin_amdgcn_readfirstlane(rows[j]) : -1;
      if (row < 0) continue;
      const float wj = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, ws[j])));
#pragma unroll
      for (int q = 0; q < VPL; ++q) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          acc[q][2 * i] = fmaf(wj, bf16lo_to_f32(buf[jj][q][i]), acc[q][2 * i]);
          acc[q][2 * i + 1] = fmaf(wj, bf16hi_to_f32(buf[jj][q][i]), acc[q][2 * i + 1]);
        }
      }
    }
  }
  // Streamed stores through a resource bounded to the output row, device scope (sc1) and
  // nontemporal: they leave no dirty lines behind and measured best of the store policies.
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(out + g * nv, 0, nv * 16, kBufferRsrcWord3);
#pragma unroll
  for (int q = 0; q < VPL; ++q) {
    if (v[q] < nv) {
      u32x4 o;
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = f32x2_to_bf16x2(acc[q][2 * i], acc[q][2 * i + 1]);
      __builtin_amdgcn_raw_buffer_store_b128(o, rs, v[q] * 16, 0, kCachePolicySc1Nt);
    }
  }
}

// unit = (token g, column chunk c). Units are numbered token-major, so one workgroup's waves
// cover at most kCombineWaves consecutive tokens; their k row indices and k gate weights are
// staged in LDS with one coalesced load per workgroup.
//
// Occupancy is capped at kCombineWavesPerSimd waves per SIMD. The compiler enforces the cap by
// reserving a larger register budget. With every resident wave holding 8 random 1 KiB gathers in
// flight, fewer waves measured faster. With 4 waves per SIMD, 16 per CU:
// * EP=64 decode: 201 -> 194 us;
// * EP=32 prefill: 3066 -> 2927 us;
// * skewed fp8: 371 -> 345 us.
// 3 waves per SIMD measured within 1% of 4. 2 waves per SIMD was too few to cover the latency.
//
// For a receive buffer of prefill size the wide form is used: 2 KiB column chunks at 2 waves per
// SIMD, the same bytes in flight per CU as 1 KiB at 4 waves but half as many concurrent read
// streams. Whole layer, two alternating runs each, combine us, 1 KiB at 4 waves against 2 KiB at
// 2 / 3 / 4 waves:
// * EP=32 prefill (15 GB of y): 2893-2896 against 2876 / 2977-2979 / 3041;
// * EP=256 (1.9 GB): 367.3-367.4 against 366.6-367.2 / 386-387 / 391-392;
// * skewed fp8 (1.9 GB): 342.3-343.2 against 343.2-344.6 / 365 / 371;
// * EP=64 decode (0.9 GB): 190.6-196.4 against 194.1-194.4 / 200 / 201.
constexpr int combine_waves_per_simd(int vpl) { return vpl == 1 ? 4 : 2; }
constexpr int64_t kWideCombineBytes = 4ll << 30;  // T*k*H*2 (the bound on y) from which the wide form runs
template <bool SMALL_K, int VPL>
__global__ void __launch_bounds__(kCombineThreads)
    __attribute__((amdgpu_waves_per_eu(combine_waves_per_simd(VPL), combine_waves_per_simd(VPL))))
    combine_kernel(const u32x4* __restrict__ y, const float* __restrict__ w, const int32_t* __restrict__ pair_row,
                   u32x4* __restrict__ out, int64_t T, int k, int nv, int pv, int chunks) {
  __shared__ int32_t rows_lds[kCombineWaves * EPL_MAX_TOPK];
  __shared__ float w_lds[kCombineWaves * EPL_MAX_TOPK];
  const int64_t units = T * chunks;
  const int lane = threadIdx.x % kWave;
  for (int64_t ub = (int64_t)blockIdx.x * kCombineWaves; ub < units; ub += (int64_t)gridDim.x * kCombineWaves) {
    const int64_t g_first = ub / chunks;
    const int64_t g_last = std::min(units - 1, ub + kCombineWaves - 1) / chunks;
    const int ntok = (int)(g_last - g_first + 1);
    __syncthreads();  // the previous iteration's readers are done with the staging buffers
    for (int i = threadIdx.x; i < ntok * k; i += kCombineThreads) {
      rows_lds[i] = pair_row[g_first * k + i];
      w_lds[i] = w[g_first * k + i];
    }
    __syncthreads();
    const int64_t unit = ub + threadIdx.x / kWave;
    if (unit >= units) continue;
    const int64_t g = unit / chunks;
    combine_unit<SMALL_K, VPL>(y, rows_lds + (g - g_first) * k, w_lds + (g - g_first) * k, out, g,
                          (int)(unit - g * chunks), k, nv, pv, lane);
  }
}

template <int VPL>
void launch_combine_vpl(const u32x4* y, const float* w, const int32_t* pair_row, u32x4* out, int64_t T, int k, int nv,
                        int pv, hipStream_t stream) {
  const int chunks = (nv + combine_cols<VPL>() - 1) / combine_cols<VPL>();
  const int64_t blocks = (T * chunks + kCombineWaves - 1) / kCombineWaves;
  const dim3 grid((unsigned)std::min<int64_t>(blocks, 1 << 30));
  if (k <= kGather)
    hipLaunchKernelGGL((combine_kernel<true, VPL>), grid, dim3(kCombineThreads), 0, stream, y, w, pair_row, out, T, k,
                       nv, pv, chunks);
  else
    hipLaunchKernelGGL((combine_kernel<false, VPL>), grid, dim3(kCombineThreads), 0, stream, y, w, pair_row, out, T, k,
                       nv, pv, chunks);
}

hipError_t launch_combine(const void* y, const float* w, const int32_t* pair_row, void* out, int64_t T, int k,
                          int H, int pitch, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  const int nv = H / 8;
  const u32x4* yv = static_cast<const u32x4*>(y);
  u32x4* ov = static_cast<u32x4*>(out);
  if (T * k * (int64_t)H * 2 >= kWideCombineBytes)
    launch_combine_vpl<2>(yv, w, pair_row, ov, T, k, nv, pitch / 8, stream);
  else
    launch_combine_vpl<1>(yv, w, pair_row, ov, T, k, nv, pitch / 8, stream);
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
