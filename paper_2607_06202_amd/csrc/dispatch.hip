// MoE dispatch on one GPU: write each token's row into the packed receive row of every valid
// (token, expert) pair.
//
// This is the paper's Token-Sending into pre-partitioned receive space (Implementation, global
// load/store; Background phase 2). Token-Reordering is fused in: the layout has already fixed
// every row, so each copy lands in its final slot.
//
// One wave per token, and every token carries at most k rows, so a contiguous token range per
// workgroup gives equal work per wave (the paper's equal token slices, Hierarchical Token-level
// Scheduling). The token row is read once with 16-byte loads and written k times with 16-byte
// nontemporal stores.
//
// The fp8 variant quantises while copying. For each 128-element block the scale is
// s = max|x| / 448, and each element is stored as q = E4M3(x / s), RNE and saturating. It
// writes the same q row and scale row to all k destinations.
#include "epl_internal.h"

namespace epl {

constexpr int kDispatchThreads = 256;
constexpr int kTokensPerBlock = kDispatchThreads / kWave;

// bf16: a row is nv = H/8 16-byte vectors; each lane holds up to VPL of them per pass.
template <int VPL>
__global__ void __launch_bounds__(kDispatchThreads)
    dispatch_bf16_kernel(const u32x4* __restrict__ x, const int32_t* __restrict__ pair_row, u32x4* __restrict__ recv,
                         int64_t T, int k, int nv, int64_t cap) {
  const int lane = threadIdx.x % kWave;
  const int64_t g = (int64_t)blockIdx.x * kTokensPerBlock + threadIdx.x / kWave;
  if (g >= T) return;
  const int my_row = lane < k ? pair_row[g * k + lane] : -1;
  const u32x4* xr = x + g * nv;
  for (int v0 = 0; v0 < nv; v0 += kWave * VPL) {
    u32x4 buf[VPL];
#pragma unroll
    for (int u = 0; u < VPL; ++u) {
      const int v = v0 + u * kWave + lane;
      if (v < nv) buf[u] = __builtin_nontemporal_load(xr + v);
    }
    for (int j = 0; j < k; ++j) {
      const int row = __builtin_amdgcn_readlane(my_row, j);
      if (row < 0 || row >= cap) continue;
      u32x4* dst = recv + (int64_t)row * nv;
#pragma unroll
      for (int u = 0; u < VPL; ++u) {
        const int v = v0 + u * kWave + lane;
        if (v < nv) __builtin_nontemporal_store(buf[u], dst + v);
      }
    }
  }
}

// fp8: a pass covers 1024 elements; lane l quantises elements [16l, 16l+16) of the pass (two
// 16-byte bf16 loads -> one 16-byte E4M3 store). A 128-element block spans 8 lanes, whose
// max is combined with three xor-shuffles. Up to PASSES passes are held in registers before
// being stored to every destination; per-block scales go through LDS so that each
// destination's scale row is stored with contiguous lanes.
template <int PASSES>
__global__ void __launch_bounds__(kDispatchThreads)
    dispatch_fp8_kernel(const u32x4* __restrict__ x, const int32_t* __restrict__ pair_row, u32x4* __restrict__ recv,
                        float* __restrict__ recv_scale, int64_t T, int k, int H, int64_t cap) {
  extern __shared__ float sc_lds[];  // [kTokensPerBlock][NB]
  const int lane = threadIdx.x % kWave;
  const int wv = threadIdx.x / kWave;
  const int64_t g = (int64_t)blockIdx.x * kTokensPerBlock + wv;
  if (g >= T) return;
  const int NB = H / 128;
  float* sc = sc_lds + wv * NB;
  const int my_row = lane < k ? pair_row[g * k + lane] : -1;
  const u32x4* xr = x + g * (H / 8);
  const int nvq = H / 16;  // 16-byte fp8 vectors per row
  const int npass = (H + 1023) / 1024;

  for (int p0 = 0; p0 < npass; p0 += PASSES) {
    u32x4 q[PASSES];
#pragma unroll
    for (int pp = 0; pp < PASSES; ++pp) {
      const int vq = (p0 + pp) * kWave + lane;  // fp8 vector index = element / 16
      const bool on = (p0 + pp < npass) && (vq < nvq);
      u32x4 a = {0, 0, 0, 0}, bv = {0, 0, 0, 0};
      if (on) {
        a = __builtin_nontemporal_load(xr + 2 * vq);
        bv = __builtin_nontemporal_load(xr + 2 * vq + 1);
      }
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
      u32x4 o = {0, 0, 0, 0};
      if (amax != 0.0f) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          o[i] = f32x4_to_e4m3x4(f[4 * i] / s, f[4 * i + 1] / s, f[4 * i + 2] / s, f[4 * i + 3] / s);
      }
      q[pp] = o;
      if (on && (lane % 8) == 0) sc[vq / 8] = s;
    }
    for (int j = 0; j < k; ++j) {
      const int row = __builtin_amdgcn_readlane(my_row, j);
      if (row < 0 || row >= cap) continue;
      u32x4* dst = recv + (int64_t)row * nvq;
#pragma unroll
      for (int pp = 0; pp < PASSES; ++pp) {
        const int vq = (p0 + pp) * kWave + lane;
        if ((p0 + pp < npass) && (vq < nvq)) __builtin_nontemporal_store(q[pp], dst + vq);
      }
    }
  }
  // Scales: the wave's own LDS writes are complete before these reads.
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  for (int j = 0; j < k; ++j) {
    const int row = __builtin_amdgcn_readlane(my_row, j);
    if (row < 0 || row >= cap) continue;
    float* dst = recv_scale + (int64_t)row * NB;
    for (int bk = lane; bk < NB; bk += kWave) __builtin_nontemporal_store(sc[bk], dst + bk);
  }
}

hipError_t launch_dispatch_bf16(const void* x, const int32_t* pair_row, void* recv, int64_t T, int k, int H,
                                int64_t cap, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  const int nv = H / 8;
  const dim3 grid((unsigned)((T + kTokensPerBlock - 1) / kTokensPerBlock));
  const u32x4* xv = static_cast<const u32x4*>(x);
  u32x4* rv = static_cast<u32x4*>(recv);
  if (nv <= kWave * 4)
    hipLaunchKernelGGL(dispatch_bf16_kernel<4>, grid, dim3(kDispatchThreads), 0, stream, xv, pair_row, rv, T, k, nv, cap);
  else
    hipLaunchKernelGGL(dispatch_bf16_kernel<14>, grid, dim3(kDispatchThreads), 0, stream, xv, pair_row, rv, T, k,
                       nv, cap);
  return hipGetLastError();
}

hipError_t launch_dispatch_fp8(const void* x, const int32_t* pair_row, void* recv, float* recv_scale, int64_t T,
                               int k, int H, int64_t cap, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  const dim3 grid((unsigned)((T + kTokensPerBlock - 1) / kTokensPerBlock));
  const size_t lds = sizeof(float) * (size_t)kTokensPerBlock * (H / 128);
  hipLaunchKernelGGL(dispatch_fp8_kernel<7>, grid, dim3(kDispatchThreads), lds, stream,
                     static_cast<const u32x4*>(x), pair_row, static_cast<u32x4*>(recv), recv_scale, T, k, H, cap);
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
