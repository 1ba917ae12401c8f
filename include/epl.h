/*
 * epl.h -- MoE expert-parallel token dispatch and combine on one MI355X (gfx950), C ABI.
 *
 * The operation (UBEP paper, Background "Deploying MoE on CM384" and the Overview):
 *   - Dispatch routes every (token, chosen expert) pair to the rank hosting that expert.
 *   - The receive space is split by (source rank, expert) and sized from per-expert token
 *     counts. The counts are turned into prefix-sum offsets ("CalCumSum", Kernel Decomposition)
 *     so that each expert's tokens end up contiguous ("Token-Reordering").
 *   - Combine gathers the expert outputs back into token order.
 *   - Senders write straight into pre-partitioned receive space (Implementation, global
 *     load/store).
 * Here all R expert-parallel ranks are virtual ranks in one GPU's HBM:
 *   - rank s sends tokens [s*Tr, (s+1)*Tr) of x;
 *   - rank d receives rows [rank_off[d], rank_off[d+1]) of the one packed receive buffer.
 *
 * Notation:
 *   R = num_ranks, E = num_experts (E % R == 0), El = E/R experts per rank;
 *   rank d owns experts [d*El, (d+1)*El);
 *   k = topk, H = hidden, Tr = tokens_per_rank, T = R*Tr;
 *   pair p = g*k + j is (token g, choice j);
 *   it is valid iff 0 <= topk_idx[p] < E, and P = number of valid pairs.
 *
 * Receive layout:
 *   - The valid pairs, stably sorted by expert id, take packed rows 0..P-1.
 *   - So rows run in (destination rank, expert, source rank, token, j) order, with no gaps.
 *   - Row r of recv, and of the expert outputs y that combine reads, starts at element r*pitch,
 *     where pitch = row_pitch, or H when row_pitch is 0. Elements [H, pitch) of a row are never
 *     read or written. The pitch moves the time in ways that depend on the row size, so it is a
 *     value to measure, not a rule: on MI355X, with H = 7168 bf16 (14 KiB rows), H + 768
 *     (15.5 KiB) took 0.6-4% off the layer at 64 ranks and 8192 tokens and changed nothing
 *     measurable at larger sizes, H + 1024 (16 KiB) made it 4% slower, and at H = 5120 every
 *     pitch above H that was tried was slower, by up to 9%.
 *
 * Conventions:
 *   - Every pointer argument is a DEVICE pointer unless stated. The caller allocates and owns
 *     every buffer, including the workspace. The library allocates nothing and keeps no state
 *     between calls.
 *   - Each call checks its arguments on the host, enqueues kernels on `stream` (a hipStream_t;
 *     NULL means the null stream) and returns without synchronising. Outputs are valid once the
 *     stream reaches that point.
 *   - Argument errors are reported BEFORE anything is enqueued.
 *   - Data-dependent anomalies are not errors: an expert id outside [0, E) is skipped and
 *     counted in *num_invalid.
 *   - Payload pointers (x, recv, y, out) must be 16-byte aligned. Index, count, weight and
 *     scale pointers must be 4-byte aligned.
 */
#ifndef EPL_H
#define EPL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define EPL_MAX_EXPERTS 1024 /* E (and therefore R) upper bound                        */
#define EPL_MAX_TOPK 32      /* k upper bound                                            */
#define EPL_MAX_HIDDEN 1048576 /* H upper bound (a row stays below 2^31 bytes)           */
#define EPL_STATIC_SCRATCH_BYTES (8u << 20) /* workspace held by the library per GPU for
                                               epl_layout_dispatch_noalloc                 */

typedef enum {
  EPL_OK = 0,
  EPL_ERR_INVALID_ARG = 1, /* bad config value, NULL where a buffer is required            */
  EPL_ERR_ALIGN = 2,       /* a pointer violates the alignment rule above                 */
  EPL_ERR_CAPACITY = 3,    /* recv_rows_cap < T*k                                          */
  EPL_ERR_WORKSPACE = 4,   /* workspace smaller than epl_workspace_bytes()                 */
  EPL_ERR_UNSUPPORTED = 5, /* fp8 payload with H % 128 != 0, unknown payload kind          */
  EPL_ERR_DEVICE = 6       /* the HIP runtime refused a launch                             */
} epl_status;

typedef enum { EPL_PAYLOAD_BF16 = 0, EPL_PAYLOAD_FP8_E4M3 = 1 } epl_payload;

typedef struct {
  int32_t num_ranks;       /* R >= 1                                                     */
  int32_t num_experts;     /* E, R <= E <= EPL_MAX_EXPERTS, E % R == 0                   */
  int32_t topk;            /* k, 1..EPL_MAX_TOPK                                         */
  int32_t hidden;          /* 8 <= H <= EPL_MAX_HIDDEN, H % 8 == 0; H % 128 == 0 for fp8 */
  int32_t tokens_per_rank; /* Tr >= 0; T*k < 2^31                                        */
  int32_t payload;         /* epl_payload: dispatch output format                        */
  int32_t row_pitch;       /* elements from one recv (and y) row to the next; 0 means H;
                              otherwise H <= row_pitch <= EPL_MAX_HIDDEN, row_pitch % 64 == 0 */
} epl_config;

/* Layout outputs: int32 device arrays, caller-allocated, all required (non-NULL).
 * send_cnt  [R*E]  send_cnt[s*E+e]: valid pairs of source rank s routed to expert e (the
 *                  per-expert token counts each source reports).
 * rank_cnt  [R*R]  rank_cnt[s*R+r]: tokens of source rank s with at least one valid pair on
 *                  rank r (tokens after per-token destination-rank dedup).
 * expert_off[E+1]  exclusive prefix sum of per-expert receive counts (CalCumSum); P = [E].
 * rank_off  [R+1]  rank_off[d] = expert_off[d*El]: rank d's rows in the packed buffer.
 * seg_off   [E*R]  seg_off[e*R+s] = expert_off[e] + sum_{s'<s} send_cnt[s'*E+e]: the
 *                  (source rank, expert) segment of the receive space.
 * tok_nranks[T]    number of distinct destination ranks of token g.
 * pair_row  [T*k]  packed receive row of pair p, or -1 if p is invalid.
 * pair_rslot[T*k]  for valid p: index of token g among the tokens of its source rank bound for
 *                  rank(topk_idx[p]), in token order (pairs of one token on one rank share
 *                  it); -1 if invalid.
 * recv_src  [T*k]  recv_src[row] = token of packed row `row`, rows 0..P-1; rows >= P untouched.
 * recv_j    [T*k]  recv_j[row] = choice index j of packed row `row`; rows >= P untouched.
 * num_invalid[1]   number of pairs whose expert id lies outside [0, E).                   */
typedef struct {
  int32_t *send_cnt;
  int32_t *rank_cnt;
  int32_t *expert_off;
  int32_t *rank_off;
  int32_t *seg_off;
  int32_t *tok_nranks;
  int32_t *pair_row;
  int32_t *pair_rslot;
  int32_t *recv_src;
  int32_t *recv_j;
  int32_t *num_invalid;
} epl_layout_buffers;

/* Bytes of device workspace epl_layout needs for `cfg` (host-only, no HIP calls). Returns 0
 * if cfg is invalid. The workspace holds per-chunk histograms and needs no initialisation. */
size_t epl_workspace_bytes(const epl_config *cfg);

/* Routing layout: per-(source rank, expert) histogram, CalCumSum prefix scans, stable slot
 * assignment and per-token destination-rank dedup (Background phases 3 and 5; Kernel
 * Decomposition: TokenCnt and CalCumSum). It takes one kernel launch up to moderate sizes
 * (see epl_layout_launches) and three beyond; both give the same outputs.
 *   topk_idx  [T*k] int32, row-major [T][k], read-only.
 *   L         output buffers above, fully overwritten (recv_src/recv_j: rows 0..P-1 only).
 *   workspace device scratch of at least epl_workspace_bytes(cfg), 4-byte aligned; its contents
 *             on entry are ignored.
 * Deterministic: identical inputs give bit-identical outputs; no atomic decides an order.    */
epl_status epl_layout(const epl_config *cfg, const int32_t *topk_idx, const epl_layout_buffers *L,
                      void *workspace, size_t workspace_bytes, void *stream);

/* Dispatch: write every valid pair's token row into its packed receive row (the paper's
 * Token-Sending into pre-partitioned receive space, with Token-Reordering fused because all
 * offsets are known before any row is written).
 *   x          [T*H] bf16 bit patterns, row-major, read-only; must not alias recv.
 *   L          a layout produced by epl_layout for the same cfg (pair_row is read).
 *   recv       recv_rows_cap rows of pitch elements (the last row may end after its H-th):
 *              bf16 (2 bytes) for EPL_PAYLOAD_BF16, or E4M3 bytes for EPL_PAYLOAD_FP8_E4M3.
 *              Elements 0..H-1 of rows 0..P-1 are written; nothing else is touched.
 *   recv_scale fp8 only: [recv_rows_cap * H/128] fp32. Scale b of a row covers columns
 *              [128b, 128b+128): s = max|x| / 448 over the block (IEEE fp32 division),
 *              q = E4M3(x / s) rounded to nearest-even with saturation to +-448, sign kept on
 *              zero, and s = 0, q = 0 for an all-zero block. Ignored (may be NULL) for bf16.
 *   recv_rows_cap  rows available in recv; must be >= T*k (T*k bounds P without a sync).
 * The rows are written in a scatter, so where recv sits in physical memory moves the time; one
 * physically contiguous block (hipExtMallocWithFlags with hipDeviceMallocContiguous) measured
 * faster on median than ordinary allocations on MI355X.                                      */
epl_status epl_dispatch(const epl_config *cfg, const void *x, const epl_layout_buffers *L, void *recv,
                        float *recv_scale, int64_t recv_rows_cap, void *stream);

/* Layout and dispatch in one call: the same outputs as epl_layout followed by epl_dispatch
 * (Kernel Decomposition: the rows are placed as the tokens are sent). For bf16 payloads with at
 * most 256 pairs per layout chunk and at most 256 experts, the layout's finalize step (stable
 * rows, dedup slots) runs inside the dispatch kernel, which saves a launch; other configs run the
 * layout and then the dispatch (see epl_layout_dispatch_launches). Arguments are those of the two
 * calls, with the same meaning, alignment and capacity rules; every status those calls can
 * return is returned before any launch. It is exactly epl_layout_counts followed by
 * epl_dispatch_rows with the same arguments.                                                 */
epl_status epl_layout_dispatch(const epl_config *cfg, const int32_t *topk_idx, const epl_layout_buffers *L,
                               void *workspace, size_t workspace_bytes, const void *x, void *recv, float *recv_scale,
                               int64_t recv_rows_cap, void *stream);

/* The two phases of epl_layout_dispatch, for callers that put work between them or time them
 * apart (Kernel Decomposition: counts and prefix sums, then sending and reordering).
 * epl_layout_counts launches the layout kernels the row kernel does not take over: histogram
 * and scan when the finalize step is fused into the row kernel, otherwise the whole layout. On
 * return (stream order) send_cnt, rank_cnt, tok_nranks and num_invalid are final; the other
 * fields of L are final only after epl_dispatch_rows. Statuses as epl_layout.
 * epl_dispatch_rows launches exactly one kernel: the fused finalize-and-send kernel, or the
 * plain dispatch kernel. It must follow epl_layout_counts on the same stream (or be ordered
 * after it) with the same cfg, topk_idx, L and workspace, none of them changed in between;
 * otherwise its outputs are undefined. Statuses as epl_layout_dispatch, all before the launch. */
epl_status epl_layout_counts(const epl_config *cfg, const int32_t *topk_idx, const epl_layout_buffers *L,
                             void *workspace, size_t workspace_bytes, void *stream);
epl_status epl_dispatch_rows(const epl_config *cfg, const int32_t *topk_idx, const epl_layout_buffers *L,
                             void *workspace, size_t workspace_bytes, const void *x, void *recv, float *recv_scale,
                             int64_t recv_rows_cap, void *stream);

/* Options of epl_layout_dispatch_decomposed. */
typedef struct {
  int32_t count_groups;      /* count workgroups; 0 picks the default (one per layout chunk, at most a
                                quarter of the workgroups the GPU holds at once); >= 0             */
  int32_t spin_limit_us;     /* bound on every wait inside the launch, microseconds; 0 = 100000     */
  int32_t test_ready_target; /* 0 in normal use. Tests of the give-up path set 2: the send workgroups
                                then wait for a value no workgroup publishes, give up after
                                spin_limit_us and store nothing, and *wait_status reports it        */
} epl_decomposed_opts;

#define EPL_WAIT_GAVE_UP_COUNT 1   /* *wait_status bit: a count workgroup stopped waiting          */
#define EPL_WAIT_GAVE_UP_SEND 2    /* *wait_status bit: a send workgroup stopped waiting           */
#define EPL_WAIT_GAVE_UP_COMBINE 4 /* *wait_status bit: a combine wave stopped waiting for a row   */
#define EPL_WAIT_SENTINEL_IN_X 8   /* *wait_status bit: an input row held EPL_SENTINEL_BF16        */

/* The reserved bf16 bit pattern of Sentinel Polling: a negative NaN with every payload bit set.
 * IEEE arithmetic on the GPU returns the canonical NaN, so computed activations do not hold it;
 * epl_sentinel_find checks a host buffer at initialisation, and the layer call reports inputs that
 * hold it (EPL_WAIT_SENTINEL_IN_X).                                                             */
#define EPL_SENTINEL_BF16 0xFFFFu

/* Layout and dispatch in ONE launch, decomposed into count and send workgroups (Kernel
 * Decomposition: some cores count tokens per expert and compute the CalCumSum offsets while the
 * others send; the senders wait point to point for the published offsets instead of a global
 * barrier). Same outputs as epl_layout_dispatch, bit for bit. Count workgroups run the layout's
 * histogram and scans; send workgroups issue the loads of their first tokens, wait for the
 * offsets, then place and write every row straight into its packed slot.
 *   bf16 payloads with at most 256 pairs per layout chunk and at most 256 experts (the geometries
 *   whose rows the send role can place per token); others return EPL_ERR_UNSUPPORTED, as does a
 *   count_groups that leaves no room for send workgroups on the GPU.
 *   workspace  as epl_layout_dispatch, and its last 1024 bytes (the synchronisation words) must be
 *              zero before the first decomposed call on it: allocate it zero-filled. Every call
 *              leaves them zero again.
 *   wait_status [1] int32, device: written when the launch completes, 0 on success, else the
 *              EPL_WAIT_* bits of the waits that expired; the outputs are then incomplete.
 * The grid is sized to what the GPU holds at once, so every workgroup a wait depends on is
 * resident; every wait is still bounded by spin_limit_us, and every workgroup runs to its end.
 * Calls on one workspace must not overlap (order them on one stream). Other arguments and
 * statuses as epl_layout_dispatch.                                                            */
epl_status epl_layout_dispatch_decomposed(const epl_config *cfg, const int32_t *topk_idx, const epl_layout_buffers *L,
                                          void *workspace, size_t workspace_bytes, const void *x, void *recv,
                                          float *recv_scale, int64_t recv_rows_cap, const epl_decomposed_opts *opts,
                                          int32_t *wait_status, void *stream);

/* The launch shape epl_layout_dispatch_decomposed would use on the current device: returns the
 * count workgroups (count_groups, or the default for 0) and stores the grid and the device's
 * co-resident capacity for the kernel; -1 for a config it does not handle. Host query, no launch. */
int epl_decomposed_plan(const epl_config *cfg, int32_t count_groups, int32_t *grid, int32_t *capacity);

/* One MoE layer in ONE launch, with identity experts: layout, dispatch, and the combine of the
 * dispatched rows (the combine reads recv itself), the combine synchronised with the dispatch per
 * row by Sentinel Polling (Data-as-Flag; Sentinel Polling variant) instead of a kernel boundary.
 * Count and send workgroups work as in epl_layout_dispatch_decomposed; combine workgroups wait for
 * the offsets, work out each token's rows, and load each 16-byte piece of a row with device-scope
 * loads until none of its elements is EPL_SENTINEL_BF16, fold it (the arithmetic of epl_combine,
 * bit for bit), and write the sentinel back over it (the reset after consumption).
 *   recv       recv_rows_cap rows of pitch bf16 elements: elements 0..H-1 of every row must hold
 *              EPL_SENTINEL_BF16 before the first call (epl_sentinel_fill over the whole buffer);
 *              each call leaves them so. No other call may write them in between.
 *   x          must not hold EPL_SENTINEL_BF16 (check with epl_sentinel_find at initialisation); a
 *              row that does is reported (EPL_WAIT_SENTINEL_IN_X) and its combine gives up.
 *   topk_w, out  as epl_combine (out [T*H] bf16 = the combine of x's rows).
 *   opts, wait_status  as epl_layout_dispatch_decomposed; count, send and combine waits are all
 *              bounded by spin_limit_us.
 * L and the workspace get the layout as epl_layout_dispatch writes it. Same shapes and statuses as
 * epl_layout_dispatch_decomposed.                                                              */
epl_status epl_layer_sentinel(const epl_config *cfg, const int32_t *topk_idx, const epl_layout_buffers *L,
                              void *workspace, size_t workspace_bytes, const void *x, void *recv, int64_t recv_rows_cap,
                              const float *topk_w, void *out, const epl_decomposed_opts *opts, int32_t *wait_status,
                              void *stream);

/* Fill kernel: n bf16 elements of buf (a multiple of 8; 16-byte aligned) set to EPL_SENTINEL_BF16. */
epl_status epl_sentinel_fill(void *buf, int64_t n, void *stream);

/* Host-only initialisation check: index of the first of n HOST bf16 values equal to
 * EPL_SENTINEL_BF16, or -1 if none (or values is NULL or n <= 0). No HIP calls.                */
int64_t epl_sentinel_find(const uint16_t *values, int64_t n);

/* The paper's other two Data-as-Flag variants (Data-as-Flag Synchronization: Token-Flag Fusion
 * and Data-for-Checksum), as alternatives to Sentinel Polling in the one-launch layer: layout,
 * dispatch and the combine of the dispatched rows (identity experts) in one launch, the combine
 * synchronised with the dispatch per 1 KiB chunk of a row. MI355X gives no 512-byte store
 * atomicity, so neither variant fuses its flag into the payload block:
 *   EPL_DAF_TOKEN_FLAG_FUSION  a send wave waits for its own row stores to complete, then stores
 *              `epoch` into the mark of every chunk it wrote; a combine wave polls the chunk's mark
 *              until it equals `epoch`, then loads the chunk.
 *   EPL_DAF_DATA_CHECKSUM      a send wave stores, with no wait, a 64-bit hash of each chunk it
 *              wrote, salted with `epoch`; a combine wave loads the chunk and its mark until the
 *              salted hash of what it loaded equals the mark. Stale or partly written data fail
 *              the comparison except with probability about 2^-64.
 *   marks      [recv_rows_cap * ceil(H/512)] uint64 device, 8-byte aligned: one word per (packed
 *              row, 1 KiB column chunk); epl_layer_marks_bytes gives its size. Its contents carry
 *              over from call to call. For EPL_DAF_TOKEN_FLAG_FUSION it must be zero-filled before
 *              the first call and every call must use an epoch no earlier call on it used; for
 *              EPL_DAF_DATA_CHECKSUM any contents will do, and each call's epoch must differ from
 *              the previous one's.
 *   epoch      nonzero (INVALID_ARG for 0).
 *   recv       receive rows as epl_layer_sentinel, with no sentinel and no fill: any contents.
 * Other arguments, outputs and statuses as epl_layer_sentinel; an unknown variant is
 * INVALID_ARG.                                                                                 */
#define EPL_DAF_TOKEN_FLAG_FUSION 1
#define EPL_DAF_DATA_CHECKSUM 2
epl_status epl_layer_data_as_flag(const epl_config *cfg, const int32_t *topk_idx, const epl_layout_buffers *L,
                                  void *workspace, size_t workspace_bytes, const void *x, void *recv,
                                  int64_t recv_rows_cap, const float *topk_w, void *out, uint64_t *marks,
                                  int32_t variant, uint64_t epoch, const epl_decomposed_opts *opts,
                                  int32_t *wait_status, void *stream);

/* Bytes of the marks buffer of epl_layer_data_as_flag for recv_rows_cap receive rows; -1 for an
 * invalid cfg or a negative count. Host-only, no HIP calls.                                    */
int64_t epl_layer_marks_bytes(const epl_config *cfg, int64_t recv_rows_cap);

/* epl_layout_dispatch without a caller workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc). Same
 * outputs, arguments, statuses and kernels as epl_layout_dispatch, except that the layout's
 * scratch is a static device array inside the library: EPL_STATIC_SCRATCH_BYTES per GPU, held from
 * the first call on that GPU until the process ends. The call allocates nothing (no hipMalloc,
 * hipFree or allocating library routine); its first call on a GPU looks up that GPU's array.
 * Limits and sharing:
 *   - returns EPL_ERR_WORKSPACE, before any launch, when epl_workspace_bytes(cfg) exceeds
 *     EPL_STATIC_SCRATCH_BYTES. 8 MiB covers every shape up to 1024 experts on 512 ranks of 64
 *     tokens (5.1 MiB) or 256 experts on 32 ranks of 8192 tokens (3.3 MiB); 1024 ranks of one
 *     expert each need 12 MiB and are refused;
 *   - every call on one GPU shares that GPU's array, which keeps the last call's contents (the
 *     kernels need no initialised scratch). Calls that overlap on one GPU (two streams, two
 *     threads) race on it and give undefined outputs: order them on one stream;
 *   - the array belongs to the device of `stream` (the current device for the null stream).    */
epl_status epl_layout_dispatch_noalloc(const epl_config *cfg, const int32_t *topk_idx, const epl_layout_buffers *L,
                                       const void *x, void *recv, float *recv_scale, int64_t recv_rows_cap,
                                       void *stream);

/* Combine: gate-weighted gather-reduce of expert output rows back into token order (the
 * paper's combine: gather expert outputs, restore token order).
 *   y       >= P rows of pitch bf16 elements (the receive layout's pitch): elements 0..H-1 of
 *           row r hold the expert result for packed row r.
 *   topk_w  [T*k] fp32 gate weights, applied as given (no renormalisation).
 *   out     [T*H] bf16. For every token g and column c:
 *             acc = +0.0f; for j = 0..k-1 with pair_row[g*k+j] >= 0:
 *                 acc = fmaf(topk_w[g*k+j], float(y[pair_row[g*k+j]][c]), acc);
 *             out[g][c] = bf16 round-to-nearest-even(acc).
 *           A token with no valid pair gets +0. out may alias x. out must not alias y.       */
epl_status epl_combine(const epl_config *cfg, const void *y, const float *topk_w, const epl_layout_buffers *L,
                       void *out, void *stream);

/* Row location (Hierarchical Token-level Scheduling, Token-level Load Partition; Algorithm 1,
 * Quaternary Search): for each position r, the expert whose cumulative range in the packed rows
 * covers r and r's offset inside that expert's rows. For a consumer that cuts the P packed rows
 * into slices (a worker or GEMM tile per slice) and needs the expert at each slice start.
 *   expert_off [E+1] int32, the layout's expert_off (from epl_layout or epl_layout_dispatch on the
 *              same stream, or ordered before it); other contents give unspecified but in-bounds
 *              results.
 *   rows       [n] int32 positions, or NULL for the positions 0..n-1.
 *   expert, offset  [n] int32 outputs: expert[i] = e with expert_off[e] <= r < expert_off[e+1]
 *              (the unique non-empty such e), offset[i] = r - expert_off[e]; both -1 when r is
 *              outside [0, P), P = expert_off[E].
 * n >= 0 (INVALID_ARG otherwise); all pointers 4-byte aligned (ALIGN). Only cfg->num_experts is
 * used beyond the config check.                                                              */
epl_status epl_locate_rows(const epl_config *cfg, const int32_t *expert_off, const int32_t *rows, int64_t n,
                           int32_t *expert, int32_t *offset, void *stream);

#define EPL_MAX_HOP_CLASSES 8 /* hop classes of epl_hop_schedule                             */

/* Hierarchical token-level schedule (Hierarchical Token-level Scheduling: Latency Homogenization;
 * Hardware-Accelerated Mapper, Expert Remapping via Logical Matrix Transposition and Token-level
 * Load Partition). For every source rank s, its valid pairs are taken expert by expert in a
 * remapped expert sequence (expert order[i] contributes send_cnt[s*E+order[i]] pairs) and cut into
 * `workers` contiguous slices whose sizes differ by at most one: worker j gets positions
 * [floor(j*m/n), floor((j+1)*m/n)) of the rank's m pairs, n = workers. For each (s, j):
 *   start_expert[s*n+j], start_offset[s*n+j]  the expert holding the slice's first position and
 *              that position's offset among the expert's pairs (Algorithm 1's lookup over the
 *              remapped cumulative counts); -1, -1 for an empty slice;
 *   class_cnt[(s*n+j)*NH+h]  the slice's pairs whose destination rank d = e / (E/R) has hop class
 *              hop_class[s*R+d] == h, 0 <= h < NH = num_classes (the per-hop loads v_{j,h}; the
 *              remap aims for v_{j,h} <= ceil(V_h / n)). A class outside [0, NH) is counted nowhere.
 * The sequence:
 *   order      [E] int32 device, the expert sequence, or NULL for the transposition: the experts
 *              laid row by row into a matrix of remap_rows rows and ceil(E/remap_rows) columns
 *              (row w holds the block of experts worker w would take without the remap), read
 *              column by column, skipping empty cells. remap_rows 0 means one row per worker
 *              (remap_rows = workers); remap_rows 1 gives the natural order 0..E-1. An order entry
 *              outside [0, E) counts as an expert with no pairs.
 *   send_cnt   [R*E] int32 device, a layout's send_cnt, or any non-negative counts whose sum per rank
 *              stays below 2^31 (other values give unspecified but in-bounds results).
 *   hop_class  [R*R] int32 device, hop class of each (source, destination rank).
 * workers >= 1 and R*workers < 2^31; 1 <= num_classes <= EPL_MAX_HOP_CLASSES; remap_rows >= 0
 * (INVALID_ARG otherwise); pointers 4-byte aligned (ALIGN). One launch of R workgroups.        */
epl_status epl_hop_schedule(const epl_config *cfg, const int32_t *send_cnt, const int32_t *order, int32_t remap_rows,
                            const int32_t *hop_class, int32_t workers, int32_t num_classes, int32_t *start_expert,
                            int32_t *start_offset, int32_t *class_cnt, void *stream);

/* Dispatch in the order of the hierarchical token-level schedule: one workgroup per (source rank
 * s, worker j) sends slice j of s's pairs, taken in the transposed expert sequence of
 * epl_hop_schedule (order NULL, same remap_rows and workers), each pair's row copied from x into
 * its packed receive row. Every worker moves floor(m/n) or ceil(m/n) rows. The output is the same
 * as epl_dispatch's, bit for bit: only which workgroup writes a row, and when, follows the
 * schedule. Each pair reads its token's row of x (k reads per token where epl_dispatch reads it
 * once), as per-pair sends do; fp8 payloads are quantised per pair, with epl_dispatch's rule.
 *   L          a layout of the same cfg: send_cnt, seg_off and recv_src are read.
 *   x, recv, recv_scale, recv_rows_cap  as epl_dispatch (recv_scale fp8 only, else ignored).
 * workers >= 1 and R*workers < 2^31, remap_rows >= 0, else INVALID_ARG; other statuses as
 * epl_dispatch.                                                                                 */
epl_status epl_dispatch_scheduled(const epl_config *cfg, const void *x, const epl_layout_buffers *L, void *recv,
                                  float *recv_scale, int64_t recv_rows_cap, int32_t remap_rows, int32_t workers,
                                  void *stream);

/* Diagnostics: apply the exact device number conversions used by epl_dispatch (fp32 ->
 * saturating E4M3) and epl_combine (fp32 -> bf16 RNE) to n values, for exhaustive checks.
 * in [n] fp32, out [n] bytes / bf16 bit patterns, 4-byte aligned; n >= 0.                   */
epl_status epl_debug_f32_to_e4m3(const float *in, uint8_t *out, int64_t n, void *stream);
epl_status epl_debug_f32_to_bf16(const float *in, uint16_t *out, int64_t n, void *stream);

/* Number of kernel launches epl_layout issues for cfg: 1 (each workgroup recomputes the global
 * counts it needs; used while T*k <= 16384, Tr*k <= 4096 and its LDS fits in 64 KiB) or 3
 * (histogram, scan, finalize). Returns -1 if cfg is invalid. Host-only, no HIP calls.        */
int epl_layout_launches(const epl_config *cfg);

/* Kernel launches epl_layout_dispatch issues for cfg: 2 (one-launch layout, dispatch),
 * 3 (histogram, scan, finalize fused into the dispatch) or 4 (three-launch layout, dispatch).
 * epl_layout_counts issues all but the last of them. Returns -1 if cfg is invalid. Host-only,
 * no HIP calls.                                                                               */
int epl_layout_dispatch_launches(const epl_config *cfg);

/* Static strings; never NULL. */
const char *epl_status_str(epl_status status);
const char *epl_version(void);

#ifdef __cplusplus
}
#endif

#endif /* EPL_H */
