// Row location: for a position r in the expert-major packed rows, the expert whose cumulative
// range covers it and r's offset inside that expert's rows (Hierarchical Token-level
// Scheduling, Token-level Load Partition; Algorithm 1, Quaternary Search). A consumer that cuts
// the P packed rows into equal slices (a grouped expert GEMM, a worker per slice) uses it to find
// where each slice starts.
//
// The paper counts list entries below three pivot experts with one vector instruction per step,
// narrowing a window of experts four ways. Here the counts below every expert are already the
// layout's expert_off, so a count is one lookup. The workgroup stages expert_off in LDS, and each
// lane searches for its own position. A step reads the three pivots' counts as three independent
// LDS loads and keeps the quarter of the window that holds the position, so a lane takes
// ceil(log4 E) dependent steps instead of log2 E.
#include "epl_internal.h"

namespace epl {

constexpr int kLocateThreads = 256;

__global__ void __launch_bounds__(kLocateThreads)
    locate_rows_kernel(const int32_t* __restrict__ expert_off, const int32_t* __restrict__ rows, int64_t n, int E,
                       int32_t* __restrict__ expert, int32_t* __restrict__ offset) {
  extern __shared__ int32_t off[];  // [E + 1]
  for (int i = threadIdx.x; i <= E; i += kLocateThreads) off[i] = expert_off[i];
  __syncthreads();
  const int P = off[E];
  for (int64_t q = (int64_t)blockIdx.x * kLocateThreads + threadIdx.x; q < n;
       q += (int64_t)gridDim.x * kLocateThreads) {
    const int64_t t = rows ? (int64_t)rows[q] : q;
    int e = -1, o = -1;
    if (t >= 0 && t < P) {
      e = quaternary_find(off, E, t);
      o = (int)(t - off[e]);
    }
    expert[q] = e;
    offset[q] = o;
  }
}

hipError_t launch_locate_rows(const int32_t* expert_off, const int32_t* rows, int64_t n, int E, int32_t* expert,
                              int32_t* offset, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((n + kLocateThreads - 1) / kLocateThreads, 4096);
  hipLaunchKernelGGL(locate_rows_kernel, dim3((unsigned)blocks), dim3(kLocateThreads), sizeof(int32_t) * (E + 1),
                     stream, expert_off, rows, n, E, expert, offset);
  return hipGetLastError();
}

}  // namespace epl
