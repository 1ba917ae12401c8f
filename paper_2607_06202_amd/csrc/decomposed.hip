// Layout and dispatch in one launch, decomposed into count and send workgroups (the paper's
// Kernel Decomposition, with its point-to-point synchronisation in place of global barriers).
//
// The three-launch path runs the layout's counts (K1), its CalCumSum scans (K2) and then the row
// kernel that places and sends, with a kernel boundary between each. Here one launch holds both
// roles, as the paper splits an NPU's vector cores into a group that counts tokens and computes
// the prefix sums and a group that sends tokens:
//   * count workgroups [0, nc) run K1 on chunks i, i + nc, ..., meet at a counter (every count
//     workgroup has finished its chunks), run the K2 items i, i + nc, ..., and count themselves
//     again; the last one publishes the ready word. They then write the expert, rank and segment
//     offsets (one slice each);
//   * send workgroups [nc, grid) issue the loads of their first tokens, wait for the ready word,
//     and then place and send rows exactly as the fused row kernel does, striding over the units.
// The count/send split nc is the knob the paper sizes by its latency model (count cores in
// proportion to the experts and inversely to the token load).
//
// Synchronisation on MI355X. Every word that one workgroup writes and another reads inside the
// launch is written with device-scope stores (ld32/st32 with C set), which need no cache
// write-back; the count role writes its per-chunk expert counts chunk-major (cnt, one contiguous
// row per chunk), because single 4-byte device-scope stores into lines that other workgroups also
// write each cost a read-modify-write in memory. A workgroup publishes by waiting for its own
// stores to complete (vmcnt), then adding to a counter with a device-scope atomic. Waiting
// workgroups poll with device-scope loads and sleep between polls; each counter and flag sits in
// a 128-byte line of its own. The count role reads what other count workgroups wrote with
// device-scope loads; a send workgroup takes one device-scope acquire after its wait (thread 0,
// passed on by the workgroup barrier) and then reads the offsets with ordinary loads.
//
// Progress. A waiting workgroup only waits for count workgroups, and the host sizes the grid to
// what the device holds at once (the occupancy of this kernel times the compute units), so every
// workgroup it waits for is resident. Every wait is still bounded (opts.spin_ticks of the 100 MHz
// real-time clock): on expiry the workgroup records a give-up bit, stores nothing more of its
// role, and runs to its end. The last workgroup to finish writes the launch's status word (zero,
// or the give-up bits) and returns every synchronisation word to zero for the next call.
#include "layout_body.h"
#include "rows_body.h"

namespace epl {

constexpr int kSyncHist = 0 * kSyncStride;    // count workgroups done with their chunks
constexpr int kSyncScan = 1 * kSyncStride;    // count workgroups done with their scan items
constexpr int kSyncReady = 2 * kSyncStride;   // 1 once every offset the send role reads is published
constexpr int kSyncExit = 3 * kSyncStride;    // workgroups done
constexpr int kSyncStatus = 4 * kSyncStride;  // give-up bits of this launch
constexpr int kGaveUpCount = 1;    // a count workgroup stopped waiting
constexpr int kGaveUpSend = 2;     // a send workgroup stopped waiting
constexpr int kGaveUpCombine = 4;  // a combine wave stopped waiting for a row
constexpr int kSentinelInX = 8;    // an input row held the sentinel

struct DecomposedArgs {
  FusedLayout F;               // what the row placement reads and writes
  int32_t* tok_nranks;         // K1 and K2 outputs and workspace
  int32_t* chunk_e;
  int32_t* chunk_r;
  int32_t* inval;
  uint32_t* fmask;
  int32_t* recv_cnt;
  int32_t* send_cnt;
  int32_t* rank_cnt;
  int32_t* seg_rel;
  int32_t* num_invalid;
  int32_t* cnt;                // [nblk][E] chunk-major expert counts
  const float* topk_w;         // the combine role (the layer variants): [T*k] weights
  u32x4* out;                  // [T][H] bf16
  uint64_t* marks;             // Token-Flag Fusion and Data-for-Checksum: [cap][cchunks] words, one per 1 KiB
  uint64_t epoch;              // this call's epoch: the flag value, or the checksum's salt
  int cchunks, nco;            // 1 KiB column chunks per row; combine workgroups
  const u32x4* x;
  u32x4* recv;
  int nv, pv, chunks;          // x row and recv pitch in 16-byte vectors; 4 KiB chunks per row
  int64_t cap;
  int nc, ns;                  // count and send workgroups
  int32_t* sync;               // [kSyncWords]
  int32_t* status;             // the call's wait status
  int64_t spin_ticks;
  int ready_target;
};

// Polls `word` with device-scope loads until it reaches `target` or `limit` ticks of the 100 MHz
// real-time clock pass. Every lane of the wave runs it with the same values.
__device__ __forceinline__ bool wait_at_least(int32_t* word, int target, int64_t limit) {
  const int64_t t0 = wall_clock64();
  while (ld32<true>(word) < target) {
    if (wall_clock64() - t0 > limit) return false;
    __builtin_amdgcn_s_sleep(2);
  }
  return true;
}

// The whole workgroup waits: thread 0 polls, the others park at the barrier. With ACQUIRE, thread
// 0 then takes a device-scope acquire (it invalidates the compute unit's L1 and the XCD's L2 of
// lines other XCDs may have changed), and the barrier passes it to the whole workgroup: its plain
// loads after the wait see everything published before the word was set.
template <bool ACQUIRE = false>
__device__ __forceinline__ bool workgroup_wait(int32_t* word, int target, int64_t limit, int32_t* flag) {
  if (threadIdx.x == 0) {
    const bool ok = wait_at_least(word, target, limit);
    if (ACQUIRE && ok) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    *flag = ok ? 1 : 0;
  }
  __syncthreads();
  const bool ok = *flag != 0;
  __syncthreads();  // every thread has read the flag before it can be rewritten
  return ok;
}

// Every thread waits for its own stores to complete; then thread 0 adds one to `counter` and
// returns the count before its add (in thread 0 only).
__device__ __forceinline__ int workgroup_publish(int32_t* counter) {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  int before = -1;
  if (threadIdx.x == 0) before = __hip_atomic_fetch_add(counter, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return before;
}

__device__ __forceinline__ void count_role(const DecomposedArgs& A, int i, int32_t* lds, int32_t* red,
                                           int32_t* scratch, int32_t* seg_start, int32_t* flag) {
  const Geom& G = A.F.G;
  for (int b = i; b < G.nblk; b += A.nc) {
    hist_chunk<true>(G, b, A.F.idx, A.tok_nranks, A.chunk_e, A.chunk_r, A.inval, A.fmask, lds, red, A.cnt);
    __syncthreads();  // the next chunk reuses the LDS
  }
  workgroup_publish(&A.sync[kSyncHist]);
  if (!workgroup_wait(&A.sync[kSyncHist], A.nc, A.spin_ticks, flag) && threadIdx.x == 0)
    atomicOr(&A.sync[kSyncStatus], kGaveUpCount);
  for (int item = i; item < G.E + G.R + 1; item += A.nc) {
    scan_item<true>(G, item, A.chunk_e, A.chunk_r, A.inval, A.recv_cnt, A.send_cnt, A.rank_cnt, A.seg_rel,
                    A.num_invalid, scratch, seg_start, A.cnt);
    __syncthreads();
  }
  const int before = workgroup_publish(&A.sync[kSyncScan]);
  if (threadIdx.x == 0 && before == A.nc - 1) {
    // Every count workgroup's stores completed before its count; publish the offsets.
    __hip_atomic_store(&A.sync[kSyncReady], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  // expert_off, rank_off and one slice of seg_off, from the published totals.
  if (workgroup_wait(&A.sync[kSyncReady], 1, A.spin_ticks, flag))
    fused_meta_block<true>(A.F, i, A.nc, lds);
  else if (threadIdx.x == 0)
    atomicOr(&A.sync[kSyncStatus], kGaveUpCount);
}

__device__ __forceinline__ bool holds_sentinel(u32x4 v);

// Places and sends the units j * 4, j * 4 + 4 * ns, ... (4 per workgroup, one per wave), as the
// fused row kernel does, after waiting for the offsets once the first unit's loads are issued.
// Measured against handing out batches of units from a launch-wide counter, with the count
// workgroups joining once their counting was done: that was slower (decode 416.7 against
// 396.8 us per layer, the Qwen3-30B shape 61.2 against 50.7 us), the counter's atomics serialising.
template <int SYNC>
__device__ __forceinline__ void publish_marks(const DecomposedArgs& A, const u32x4* buf, const bool* on, int my_row,
                                              int c, int k, int lane);

template <bool BUF_X, int SYNC>
__device__ __forceinline__ void send_role(const DecomposedArgs& A, int j, int32_t* lds, int32_t* flag) {
  const int lane = threadIdx.x % kWave;
  const int w = threadIdx.x / kWave;
  const int k = A.F.G.k;
  int32_t* rows_lds = lds;  // [kWavesPerBlock][k]
  int32_t* hist = lds + kWavesPerBlock * EPL_MAX_TOPK + w * (A.F.G.E + A.F.G.R);
  const int64_t units = A.F.G.T * A.chunks;
  const int64_t stride = (int64_t)A.ns * kWavesPerBlock;
  bool waited = false, gave_up = false;
  // The loop bound depends on the workgroup's first unit only, so every wave runs the same
  // iterations and reaches the same barriers.
  for (int64_t ub = (int64_t)j * kWavesPerBlock; ub < units && !gave_up; ub += stride) {
    const int64_t g_first = ub / A.chunks;
    const int64_t g_last = std::min(units - 1, ub + kWavesPerBlock - 1) / A.chunks;
    const int64_t u = ub + w;
    const bool active = u < units;
    const int64_t g = (active ? u : units - 1) / A.chunks;
    const int c = (int)((active ? u : units - 1) - g * A.chunks);
    dispatch_bf16_unit<BUF_X>(
        A.x,
        [&] {
          if (!waited) {  // the first unit's loads of x are in flight while the offsets arrive
            waited = true;
            gave_up = !workgroup_wait<true>(&A.sync[kSyncReady], A.ready_target, A.spin_ticks, flag);
            if (gave_up && threadIdx.x == 0) atomicOr(&A.sync[kSyncStatus], kGaveUpSend);
          }
          if (gave_up) return -1;  // uniform over the workgroup: nothing is stored
          if (w <= g_last - g_first) {
            const int r = token_rows<false>(A.F, g_first + w, true, hist, lane);
            if (lane < k) rows_lds[w * k + lane] = r;
          }
          __syncthreads();
          const int r = lane < k ? rows_lds[(g - g_first) * k + lane] : -1;
          __syncthreads();  // every wave has its rows before the next iteration rewrites them
          return r;
        },
        A.recv, g, c, k, A.nv, A.pv, A.cap, lane, active,
        [&](const u32x4* buf, const bool* on) {
          if constexpr (SYNC == kDafSentinel) {
            bool seen = false;
#pragma unroll
            for (int q = 0; q < kBf16VPL; ++q) seen |= on[q] && holds_sentinel(buf[q]);
            if (__ballot(seen) != 0 && lane == 0) atomicOr(&A.sync[kSyncStatus], kSentinelInX);
          }
        },
        [&](const u32x4* buf, const bool* on, int my_row) {
          if constexpr (SYNC == kDafFlag || SYNC == kDafChecksum) publish_marks<SYNC>(A, buf, on, my_row, c, k, lane);
        });
  }
}

// ------------------------------------------------------------------------ Sentinel Polling
// The layer variant adds combine workgroups that gather the dispatched rows (identity experts:
// the combine reads the receive buffer itself) while the send workgroups are still writing them,
// with no barrier in between: the paper's Sentinel Polling (Data-as-Flag). Every receive row holds
// the reserved bf16 pattern EPL_SENTINEL_BF16 (a negative NaN with every payload bit set, which
// arithmetic does not produce) in every element before the send role writes it. A combine lane
// loads its 16 bytes of a row with device-scope loads until none of its 8 elements is the
// sentinel. MI355X gives no 512-byte store atomicity, so the check is per element rather than on
// a leading flag field: a row counts as arrived, for one lane, exactly when each of that lane's
// elements has been written, whatever the order or granularity of the stores. After folding a
// row the lane writes the sentinel back over what it read, so the buffer is ready for the next
// layer (the paper's reset after consumption). The send role checks every input vector for the
// sentinel and reports one (a row that carries it would never count as arrived).
constexpr uint32_t kSentinelPair = 0xFFFFFFFFu;  // two bf16 sentinels

__device__ __forceinline__ bool holds_sentinel(u32x4 v) {
  bool any = false;
#pragma unroll
  for (int i = 0; i < 4; ++i) any |= ((v[i] & 0xFFFFu) == 0xFFFFu) | ((v[i] >> 16) == 0xFFFFu);
  return any;
}

// Device-scope 16-byte load and store of vector v of a row of nv vectors.
__device__ __forceinline__ u32x4 load_vec_dev(const u32x4* row, int nv, int v) {
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(const_cast<u32x4*>(row), 0, nv * 16, kBufferRsrcWord3);
  return __builtin_amdgcn_raw_buffer_load_b128(r, v * 16, 0, kCachePolicySc1);
}

// Loads lane's vector v of `row` until no lane of the wave sees a sentinel in its vector, or
// `limit` ticks pass (false). The loop condition is wave-uniform.
__device__ __forceinline__ bool poll_vec(const u32x4* row, int nv, int v, u32x4& val, int64_t limit) {
  val = load_vec_dev(row, nv, v);
  if (__ballot(holds_sentinel(val)) == 0) return true;
  const int64_t t0 = wall_clock64();
  while (true) {
    __builtin_amdgcn_s_sleep(1);
    if (holds_sentinel(val)) val = load_vec_dev(row, nv, v);
    if (__ballot(holds_sentinel(val)) == 0) return true;
    if (wall_clock64() - t0 > limit) return false;
  }
}

// ------------------------------------------------------------------------ Token-Flag Fusion, Data-for-Checksum
// The paper's other two Data-as-Flag variants, for a GPU without multi-word store atomicity. Both
// keep one 64-bit word per (packed row, 1 KiB column chunk) in `marks`, beside the rows, and an
// epoch that the caller changes on every call, so nothing has to be reset between layers.
// * Token-Flag Fusion: the paper stores a flag field and the payload in one atomic 512-byte block.
//   Here a send wave waits until its own device-scope row stores are complete (vmcnt), then stores
//   the epoch into the marks of the chunks it wrote; a combine wave polls the mark until it holds
//   the epoch and only then loads the chunk. The wait on the sender is what the fused flag avoids
//   on the paper's fabric.
// * Data-for-Checksum: the paper's receiver waits for a checksum of the batch's leading markers,
//   written after the batch. Without block atomicity a marker does not vouch for the rest of its
//   block, so the checksum here covers every byte of its 1 KiB chunk: a 64-bit hash of the chunk,
//   salted with the epoch. The send wave stores it with no wait at all; a combine wave loads the
//   chunk and the mark and accepts the chunk when the hash of what it loaded, salted the same way,
//   equals the mark (else it loads both again). Stale data, a stale mark, or a chunk only partly
//   written all fail the comparison except with probability about 2^-64.
__device__ __forceinline__ uint64_t ld64_dev(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st64_dev(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The SplitMix64 output function (Steele, Lea and Flood, "Fast splittable pseudorandom number
// generators", OOPSLA 2014): a bijective 64-bit mixer.
__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// One lane's 16 bytes at lane position `lane` of its chunk, mixed; lanes outside the row give 0.
__device__ __forceinline__ uint64_t lane_hash(u32x4 v, bool on, int lane) {
  const uint64_t a = (uint64_t)v[0] | ((uint64_t)v[1] << 32);
  const uint64_t b = (uint64_t)v[2] | ((uint64_t)v[3] << 32);
  return on ? mix64(a ^ mix64(b + 0x9E3779B97F4A7C15ull * (uint64_t)(lane + 1))) : 0;
}

// XOR over the wave's 64 lanes; every lane returns the total.
__device__ __forceinline__ uint64_t wave_xor64(uint64_t h) {
  int lo = (int)(uint32_t)h, hi = (int)(uint32_t)(h >> 32);
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) {
    lo ^= __shfl_xor(lo, m, kWave);
    hi ^= __shfl_xor(hi, m, kWave);
  }
  return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

__device__ __forceinline__ uint64_t epoch_salt(uint64_t epoch) { return mix64(epoch ^ 0x5851F42D4C957F2Dull); }

// After a send wave's stores of unit (token, 4 KiB chunk c): the marks of the kBf16VPL 1 KiB
// chunks it wrote, for each of the token's destination rows (my_row in lanes 0..k-1).
template <int SYNC>
__device__ __forceinline__ void publish_marks(const DecomposedArgs& A, const u32x4* buf, const bool* on, int my_row,
                                              int c, int k, int lane) {
  uint64_t val[kBf16VPL];
  if constexpr (SYNC == kDafChecksum) {
    const uint64_t salt = epoch_salt(A.epoch);
#pragma unroll
    for (int u = 0; u < kBf16VPL; ++u) val[u] = wave_xor64(lane_hash(buf[u], on[u], lane)) ^ salt;
  } else {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's device-scope row stores are complete
#pragma unroll
    for (int u = 0; u < kBf16VPL; ++u) val[u] = A.epoch;
  }
  // Index i = j * kBf16VPL + u names destination j's chunk u; lanes take them in rounds of 64.
  for (int base = 0; base < k * kBf16VPL; base += kWave) {
    const int i = base + lane;
    const int j = i / kBf16VPL, u = i % kBf16VPL;
    const int row = __shfl(my_row, j < k ? j : 0, kWave);
    uint64_t m = val[0];
#pragma unroll
    for (int q = 1; q < kBf16VPL; ++q) m = u == q ? val[q] : m;
    const int cc = c * kBf16VPL + u;
    if (j < k && row >= 0 && row < A.cap && cc < A.cchunks) st64_dev(&A.marks[(int64_t)row * A.cchunks + cc], m);
  }
}

// Token-Flag Fusion: polls the chunk's mark until it holds the epoch, then loads the lane's vector.
// The loop condition is wave-uniform (one mark per wave).
__device__ __forceinline__ bool poll_flag(const uint64_t* mark, uint64_t epoch, const u32x4* row, int nv, int v,
                                          u32x4& val, int64_t limit) {
  if (ld64_dev(mark) != epoch) {
    const int64_t t0 = wall_clock64();
    do {
      if (wall_clock64() - t0 > limit) return false;
      __builtin_amdgcn_s_sleep(1);
    } while (ld64_dev(mark) != epoch);
  }
  val = load_vec_dev(row, nv, v);
  return true;
}

// Data-for-Checksum: loads the lane's vector and the chunk's mark until the salted hash of the
// wave's loaded chunk equals the mark. The comparison is wave-uniform.
__device__ __forceinline__ bool poll_checksum(const uint64_t* mark, uint64_t salt, const u32x4* row, int nv, int v,
                                              bool on, int lane, u32x4& val, int64_t limit) {
  int64_t t0 = -1;
  while (true) {
    const uint64_t m = ld64_dev(mark);
    val = load_vec_dev(row, nv, v);
    if ((wave_xor64(lane_hash(val, on, lane)) ^ salt) == m) return true;
    if (t0 < 0)
      t0 = wall_clock64();
    else if (wall_clock64() - t0 > limit)
      return false;
    __builtin_amdgcn_s_sleep(1);
  }
}

// Combine units (token g, 1 KiB column chunk c): one wave per unit, waves iterating on their own.
// Each wave works out its token's rows as the send role does (no metadata written), then folds
// the valid rows in j order, acc = fmaf(w_j, y_j, acc) from +0, bf16 round-to-nearest-even, as
// the combine kernel does.
template <int SYNC>
__device__ __forceinline__ void combine_role(const DecomposedArgs& A, int ci, int32_t* lds, int32_t* flag) {
  const Geom& G = A.F.G;
  const int lane = threadIdx.x % kWave;
  const int w = threadIdx.x / kWave;
  const int k = G.k;
  int32_t* hist = lds + kWavesPerBlock * EPL_MAX_TOPK + w * (G.E + G.R);
  if (!workgroup_wait<true>(&A.sync[kSyncReady], A.ready_target, A.spin_ticks, flag)) {
    if (threadIdx.x == 0) atomicOr(&A.sync[kSyncStatus], kGaveUpCombine);
    return;
  }
  const int nv = A.nv;
  const int64_t units = G.T * A.cchunks;
  const int64_t stride = (int64_t)A.nco * kWavesPerBlock;
  const u32x4* y = A.recv;
  const uint64_t salt = epoch_salt(A.epoch);
  for (int64_t u = (int64_t)ci * kWavesPerBlock + w; u < units; u += stride) {
    const int64_t g = u / A.cchunks;
    const int c = (int)(u - g * A.cchunks);
    const int rows = token_rows<false>(A.F, g, false, hist, lane);
    const int v = c * kWave + lane;
    const bool on = v < nv;
    const int vl = min(v, nv - 1);
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
    bool arrived = true;
    for (int j = 0; j < k; ++j) {
      const int row = __builtin_amdgcn_readlane(rows, j);
      if (row < 0) continue;
      const float wj = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(
                                                      __builtin_bit_cast(int, A.topk_w[g * k + j])));
      const u32x4* yr = y + (int64_t)row * A.pv;
      u32x4 val;
      bool got;
      if constexpr (SYNC == kDafFlag)
        got = poll_flag(A.marks + (int64_t)row * A.cchunks + c, A.epoch, yr, nv, vl, val, A.spin_ticks);
      else if constexpr (SYNC == kDafChecksum)
        got = poll_checksum(A.marks + (int64_t)row * A.cchunks + c, salt, yr, nv, vl, on, lane, val, A.spin_ticks);
      else
        got = poll_vec(yr, nv, vl, val, A.spin_ticks);
      if (!got) {
        arrived = false;
        break;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[2 * i] = fmaf(wj, bf16lo_to_f32(val[i]), acc[2 * i]);
        acc[2 * i + 1] = fmaf(wj, bf16hi_to_f32(val[i]), acc[2 * i + 1]);
      }
      if (SYNC == kDafSentinel && on) {  // consumed: back to the sentinel for the next layer
        const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(const_cast<u32x4*>(yr), 0, nv * 16,
                                                                           kBufferRsrcWord3);
        const u32x4 s = {kSentinelPair, kSentinelPair, kSentinelPair, kSentinelPair};
        __builtin_amdgcn_raw_buffer_store_b128(s, r, v * 16, 0, kCachePolicySc1);
      }
    }
    if (!arrived) {  // wave-uniform: stop, store nothing more
      if (lane == 0) atomicOr(&A.sync[kSyncStatus], kGaveUpCombine);
      break;
    }
    if (on) {
      u32x4 o;
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = f32x2_to_bf16x2(acc[2 * i], acc[2 * i + 1]);
      const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(A.out + g * nv, 0, nv * 16, kBufferRsrcWord3);
      __builtin_amdgcn_raw_buffer_store_b128(o, r, v * 16, 0, kCachePolicySc1Nt);
    }
  }
}

// The last workgroup to finish writes the status word and zeroes the synchronisation words. Every
// other workgroup has passed all its waits by then.
__device__ __forceinline__ void finish(const DecomposedArgs& A) {
  const int before = workgroup_publish(&A.sync[kSyncExit]);
  if (threadIdx.x == 0 && before == (int)gridDim.x - 1) {
    st32<true>(A.status, ld32<true>(&A.sync[kSyncStatus]));
    for (int i = 0; i < kSyncWords; i += kSyncStride) st32<true>(&A.sync[i], 0);
  }
}

template <bool BUF_X, int SYNC>
__global__ void __launch_bounds__(kLayoutThreads) decomposed_kernel(DecomposedArgs A) {
  static_assert(kDispatchThreads == kLayoutThreads, "both roles run in 256-thread workgroups");
  extern __shared__ int32_t lds[];
  __shared__ int32_t red[kLayoutWaves];
  __shared__ int32_t scratch[kLayoutWaves];
  __shared__ int32_t seg_start[EPL_MAX_EXPERTS + 1];
  __shared__ int32_t flag;
  if ((int)blockIdx.x < A.nc)
    count_role(A, (int)blockIdx.x, lds, red, scratch, seg_start, &flag);
  else if (SYNC == kDafNone || (int)blockIdx.x < A.nc + A.ns)
    send_role<BUF_X, SYNC>(A, (int)blockIdx.x - A.nc, lds, &flag);
  else
    combine_role<SYNC>(A, (int)blockIdx.x - A.nc - A.ns, lds, &flag);
  finish(A);
}

// ------------------------------------------------------------------------ host
namespace {

template <bool BUF_X>
void launch_variant(int sync, dim3 grid, dim3 block, size_t lds, hipStream_t stream, const DecomposedArgs& A) {
  switch (sync) {
    case kDafSentinel:
      hipLaunchKernelGGL((decomposed_kernel<BUF_X, kDafSentinel>), grid, block, lds, stream, A);
      break;
    case kDafFlag:
      hipLaunchKernelGGL((decomposed_kernel<BUF_X, kDafFlag>), grid, block, lds, stream, A);
      break;
    case kDafChecksum:
      hipLaunchKernelGGL((decomposed_kernel<BUF_X, kDafChecksum>), grid, block, lds, stream, A);
      break;
    default:
      hipLaunchKernelGGL((decomposed_kernel<BUF_X, kDafNone>), grid, block, lds, stream, A);
  }
}

size_t decomposed_lds_bytes(const Geom& g) {
  const size_t hist = (size_t)g.E + g.R + kMaxChunkPairs;                       // K1
  const size_t rows = (size_t)kWavesPerBlock * (EPL_MAX_TOPK + g.E + g.R);      // row placement
  const size_t meta = (size_t)g.E + 1;                                           // offsets
  return sizeof(int32_t) * std::max(hist, std::max(rows, meta));
}

}  // namespace

template <bool BUF_X, int SYNC>
static hipError_t occupancy(int* per_cu, size_t lds) {
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(per_cu, decomposed_kernel<BUF_X, SYNC>, kLayoutThreads, lds);
}

template <bool BUF_X>
static hipError_t occupancy_of(int sync, int* per_cu, size_t lds) {
  switch (sync) {
    case kDafSentinel: return occupancy<BUF_X, kDafSentinel>(per_cu, lds);
    case kDafFlag: return occupancy<BUF_X, kDafFlag>(per_cu, lds);
    case kDafChecksum: return occupancy<BUF_X, kDafChecksum>(per_cu, lds);
    default: return occupancy<BUF_X, kDafNone>(per_cu, lds);
  }
}

hipError_t plan_decomposed(const Geom& g, int H, int count_groups, int sync, DecomposedPlan* plan) {
  const bool layer = sync != kDafNone;
  int dev = 0, cus = 0, per_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  const bool buf_x = g.T * (int64_t)H * 2 >= kBufferLoadXBytes;
  const size_t lds = decomposed_lds_bytes(g);
  if (e == hipSuccess)
    e = buf_x ? occupancy_of<true>(sync, &per_cu, lds) : occupancy_of<false>(sync, &per_cu, lds);
  if (e != hipSuccess) return e;
  plan->capacity = per_cu * cus;
  // Default split: one count workgroup per layout chunk, at most a quarter of what the device
  // holds at once.
  int nc = count_groups > 0 ? count_groups : std::min(g.nblk, std::max(1, plan->capacity / 4));
  plan->count_groups = nc;
  const int nv = H / 8;
  const int chunks = (nv + kBf16Cols - 1) / kBf16Cols;
  const int64_t unit_blocks = (g.T * chunks + kWavesPerBlock - 1) / kWavesPerBlock;
  const int64_t room = plan->capacity - nc;
  if (!layer) {
    plan->send_groups = (int)std::max<int64_t>(1, std::min<int64_t>(room, unit_blocks));
    plan->combine_groups = 0;
  } else {
    // The rest split evenly between send and combine workgroups, each no more than it has units for.
    const int cchunks = (nv + kWave - 1) / kWave;
    const int64_t combine_blocks = (g.T * cchunks + kWavesPerBlock - 1) / kWavesPerBlock;
    plan->send_groups = (int)std::max<int64_t>(1, std::min<int64_t>(room / 2, unit_blocks));
    plan->combine_groups = (int)std::max<int64_t>(1, std::min<int64_t>(room - plan->send_groups, combine_blocks));
  }
  plan->grid = nc + plan->send_groups + plan->combine_groups;
  return hipSuccess;
}

hipError_t launch_decomposed(const Geom& g, const int32_t* idx, int32_t* ws, const epl_layout_buffers& L,
                             const void* x, void* recv, int H, int pitch, int64_t cap, const DecomposedOpts& opts,
                             int32_t* wait_status, hipStream_t stream, int sync, const float* topk_w, void* out,
                             uint64_t* marks, uint64_t epoch) {
  DecomposedPlan plan;
  hipError_t e = plan_decomposed(g, H, opts.count_groups, sync, &plan);
  if (e != hipSuccess) return e;
  if (plan.grid > plan.capacity) return hipErrorLaunchOutOfResources;  // refused on the host before this
  const WsLayout wl = ws_layout(g);
  DecomposedArgs A;
  A.F = FusedLayout{g,          idx,          ws + wl.chunk_e, ws + wl.chunk_r,
                    ws + wl.recv_cnt, ws + wl.seg_rel, reinterpret_cast<const uint32_t*>(ws + wl.fmask),
                    L.expert_off, L.rank_off,     L.seg_off,       L.pair_row,
                    L.pair_rslot, L.recv_src,     L.recv_j};
  A.tok_nranks = L.tok_nranks;
  A.chunk_e = ws + wl.chunk_e;
  A.chunk_r = ws + wl.chunk_r;
  A.inval = ws + wl.inval;
  A.fmask = reinterpret_cast<uint32_t*>(ws + wl.fmask);
  A.recv_cnt = ws + wl.recv_cnt;
  A.send_cnt = L.send_cnt;
  A.rank_cnt = L.rank_cnt;
  A.seg_rel = ws + wl.seg_rel;
  A.num_invalid = L.num_invalid;
  A.cnt = ws + wl.cnt;
  A.topk_w = topk_w;
  A.out = static_cast<u32x4*>(out);
  A.marks = marks;
  A.epoch = epoch;
  A.x = static_cast<const u32x4*>(x);
  A.recv = static_cast<u32x4*>(recv);
  A.nv = H / 8;
  A.pv = pitch / 8;
  A.chunks = (A.nv + kBf16Cols - 1) / kBf16Cols;
  A.cchunks = (A.nv + kWave - 1) / kWave;
  A.cap = cap;
  A.nc = plan.count_groups;
  A.ns = plan.send_groups;
  A.nco = plan.combine_groups;
  A.sync = ws + wl.sync;
  A.status = wait_status;
  A.spin_ticks = opts.spin_ticks;
  A.ready_target = opts.ready_target;
  const size_t lds = decomposed_lds_bytes(g);
  const bool buf_x = g.T * (int64_t)H * 2 >= kBufferLoadXBytes;
  const dim3 grid(plan.grid), block(kLayoutThreads);
  if (buf_x)
    launch_variant<true>(sync, grid, block, lds, stream, A);
  else
    launch_variant<false>(sync, grid, block, lds, stream, A);
  return hipGetLastError();
}

// The fill kernel: every 16-byte vector of the buffer set to sentinels.
__global__ void sentinel_fill_kernel(u32x4* __restrict__ buf, int64_t nvec) {
  const u32x4 s = {kSentinelPair, kSentinelPair, kSentinelPair, kSentinelPair};
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nvec; i += (int64_t)gridDim.x * blockDim.x)
    buf[i] = s;
}

hipError_t launch_sentinel_fill(void* buf, int64_t nvec, hipStream_t stream) {
  if (nvec == 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((nvec + 255) / 256, 8192);
  hipLaunchKernelGGL(sentinel_fill_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, static_cast<u32x4*>(buf),
                     nvec);
  return hipGetLastError();
}

}  // namespace epl
