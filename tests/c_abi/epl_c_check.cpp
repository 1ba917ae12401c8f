// Standalone C++ consumer of the C ABI in include/epl.h: no Python, no torch. It allocates
// device buffers with the HIP runtime, runs layout -> dispatch -> combine, the row location, the
// hierarchical schedule and the dispatch in its order, and the one-launch layer synchronised by
// Token-Flag Fusion and by Data-for-Checksum on its own stream, and compares every output
// with the CPU oracle (oracle/liboracle.so, test
// infrastructure), then checks that host-detectable errors are reported before anything is launched.
// Prints "c abi check ok" and exits 0 on success; prints the first difference and exits 1.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "epl.h"

extern "C" {  // the oracle's entry points (plain C, no header shared with the library)
int eplref_layout(int R, int E, int k, int Tr, const int32_t* idx, int32_t* send_cnt, int32_t* rank_cnt,
                  int32_t* expert_off, int32_t* rank_off, int32_t* seg_off, int32_t* tok_nranks, int32_t* pair_row,
                  int32_t* pair_rslot, int32_t* recv_src, int32_t* recv_j, int32_t* num_invalid);
void eplref_dispatch_bf16(int64_t T, int k, int H, const uint16_t* x, const int32_t* pair_row, uint16_t* recv);
void eplref_dispatch_fp8(int64_t T, int k, int H, const uint16_t* x, const int32_t* pair_row, uint8_t* recv,
                         float* recv_scale);
void eplref_combine(int64_t T, int k, int H, const uint16_t* y, const float* w, const int32_t* pair_row,
                    const int64_t* tokens, int64_t n_tokens, uint16_t* out);
void eplref_locate_rows(int E, const int32_t* expert_off, int64_t n, const int32_t* rows, int32_t* expert,
                        int32_t* offset);
void eplref_transposed_order(int E, int rows, int32_t* order);
void eplref_hop_schedule(int R, int E, int n, int NH, const int32_t* send_cnt, const int32_t* order,
                         const int32_t* hop, int32_t* start_expert, int32_t* start_offset, int32_t* counts);
}

#define HIP_OK(x)                                                                              \
  do {                                                                                         \
    hipError_t e_ = (x);                                                                       \
    if (e_ != hipSuccess) {                                                                    \
      std::printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__);               \
      std::exit(1);                                                                            \
    }                                                                                          \
  } while (0)

namespace {

uint64_t splitmix(uint64_t& s) {
  uint64_t z = (s += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

template <typename T>
T* dev_copy(const std::vector<T>& h) {
  T* d = nullptr;
  HIP_OK(hipMalloc(&d, std::max<size_t>(1, h.size()) * sizeof(T)));
  if (!h.empty()) HIP_OK(hipMemcpy(d, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice));
  return d;
}

template <typename T>
std::vector<T> host_copy(const T* d, size_t n) {
  std::vector<T> h(n);
  if (n) HIP_OK(hipMemcpy(h.data(), d, n * sizeof(T), hipMemcpyDeviceToHost));
  return h;
}

template <typename T>
bool same(const char* what, const std::vector<T>& got, const std::vector<T>& want, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (std::memcmp(&got[i], &want[i], sizeof(T)) != 0) {
      std::printf("%s differs at %zu\n", what, i);
      return false;
    }
  return true;
}

struct Case {
  int R, E, k, Tr, H;
  epl_payload payload;
  int pitch;  // epl_config.row_pitch (0: packed rows)
};

// Rows 0..P-1 of a [rows][pitch] buffer, without the gaps.
template <typename T>
std::vector<T> payload_rows(const std::vector<T>& buf, size_t P, int H, int pitch) {
  std::vector<T> out(P * H);
  for (size_t r = 0; r < P; ++r) std::memcpy(&out[r * H], &buf[r * pitch], H * sizeof(T));
  return out;
}

// How layout and dispatch are called: epl_layout then epl_dispatch, one epl_layout_dispatch
// call, or its two phases epl_layout_counts then epl_dispatch_rows.
enum Mode { kSeparate, kOneCall, kTwoPhases };
const char* const kModeName[] = {"epl_layout + epl_dispatch", "epl_layout_dispatch",
                                 "epl_layout_counts + epl_dispatch_rows"};

bool run_case(const Case& c, uint64_t seed, hipStream_t stream, Mode mode) {
  const int64_t T = (int64_t)c.R * c.Tr, Tk = T * c.k;
  const bool fp8 = c.payload == EPL_PAYLOAD_FP8_E4M3;
  std::vector<int32_t> idx(Tk);
  for (auto& v : idx) v = (int32_t)(splitmix(seed) % (uint64_t)(c.E + 2)) - 1;  // duplicates and invalid ids
  std::vector<uint16_t> x((size_t)T * c.H), y((size_t)Tk * c.H);
  for (auto& v : x) v = (uint16_t)(0x3C00 + (splitmix(seed) % 0x0800) - 0x0400) ^ (uint16_t)((splitmix(seed) & 1) << 15);
  for (auto& v : y) v = (uint16_t)(0x3F00 + (splitmix(seed) % 0x0200) - 0x0100);
  std::vector<float> w(Tk);
  for (auto& v : w) v = (float)(splitmix(seed) % 1000) / 1000.0f - 0.25f;

  epl_config cfg{c.R, c.E, c.k, c.H, c.Tr, c.payload, c.pitch};
  const int PP = c.pitch ? c.pitch : c.H;  // elements from one recv (and y) row to the next
  std::vector<uint16_t> y_pitched((size_t)Tk * PP, 0x7FC3);  // NaN patterns in the gaps
  for (int64_t r = 0; r < Tk; ++r) std::memcpy(&y_pitched[r * PP], &y[r * c.H], c.H * 2);
  // reference
  std::vector<int32_t> r_send(c.R * c.E), r_rank(c.R * c.R), r_eoff(c.E + 1), r_roff(c.R + 1), r_seg(c.E * c.R),
      r_ntok(T), r_row(Tk), r_slot(Tk), r_src(Tk), r_j(Tk), r_inv(1);
  if (eplref_layout(c.R, c.E, c.k, c.Tr, idx.data(), r_send.data(), r_rank.data(), r_eoff.data(), r_roff.data(),
                    r_seg.data(), r_ntok.data(), r_row.data(), r_slot.data(), r_src.data(), r_j.data(), r_inv.data()) != 0) {
    std::printf("oracle rejected the case\n");
    return false;
  }
  const int32_t P = r_eoff[c.E];

  // device
  int32_t* d_idx = dev_copy(idx);
  std::vector<int32_t*> d_out;
  const size_t sizes[] = {(size_t)c.R * c.E, (size_t)c.R * c.R, (size_t)c.E + 1, (size_t)c.R + 1, (size_t)c.E * c.R,
                          (size_t)T,         (size_t)Tk,        (size_t)Tk,      (size_t)Tk,      (size_t)Tk,
                          1};
  for (size_t n : sizes) {
    int32_t* p = nullptr;
    HIP_OK(hipMalloc(&p, std::max<size_t>(n, 1) * 4));
    d_out.push_back(p);
  }
  epl_layout_buffers L{d_out[0], d_out[1], d_out[2], d_out[3], d_out[4], d_out[5],
                       d_out[6], d_out[7], d_out[8], d_out[9], d_out[10]};
  const size_t ws_bytes = epl_workspace_bytes(&cfg);
  void* ws = nullptr;
  HIP_OK(hipMalloc(&ws, ws_bytes));
  uint16_t* d_x = dev_copy(x);
  uint16_t* d_y = dev_copy(y_pitched);
  float* d_w = dev_copy(w);
  void* d_recv = nullptr;
  float* d_scale = nullptr;
  HIP_OK(hipMalloc(&d_recv, (size_t)std::max<int64_t>(Tk, 1) * PP * (fp8 ? 1 : 2)));
  if (fp8) HIP_OK(hipMalloc(&d_scale, (size_t)std::max<int64_t>(Tk, 1) * (c.H / 128) * sizeof(float)));
  uint16_t* d_o = nullptr;
  HIP_OK(hipMalloc(&d_o, (size_t)std::max<int64_t>(T, 1) * c.H * 2));

  bool ok;
  if (mode == kOneCall)
    ok = epl_layout_dispatch(&cfg, d_idx, &L, ws, ws_bytes, d_x, d_recv, d_scale, Tk, stream) == EPL_OK;
  else if (mode == kTwoPhases)
    ok = epl_layout_counts(&cfg, d_idx, &L, ws, ws_bytes, stream) == EPL_OK &&
         epl_dispatch_rows(&cfg, d_idx, &L, ws, ws_bytes, d_x, d_recv, d_scale, Tk, stream) == EPL_OK;
  else
    ok = epl_layout(&cfg, d_idx, &L, ws, ws_bytes, stream) == EPL_OK &&
         epl_dispatch(&cfg, d_x, &L, d_recv, d_scale, Tk, stream) == EPL_OK;
  ok = ok && epl_combine(&cfg, d_y, d_w, &L, d_o, stream) == EPL_OK;
  if (!ok) std::printf("a call returned an error status\n");
  HIP_OK(hipStreamSynchronize(stream));

  const std::vector<int32_t>* refs[] = {&r_send, &r_rank, &r_eoff, &r_roff, &r_seg, &r_ntok, &r_row, &r_slot};
  const char* names[] = {"send_cnt", "rank_cnt", "expert_off", "rank_off", "seg_off", "tok_nranks", "pair_row",
                         "pair_rslot"};
  for (int i = 0; ok && i < 8; ++i) ok = same(names[i], host_copy(d_out[i], sizes[i]), *refs[i], sizes[i]);
  ok = ok && same("recv_src", host_copy(d_out[8], P), r_src, P) && same("recv_j", host_copy(d_out[9], P), r_j, P) &&
       same("num_invalid", host_copy(d_out[10], 1), r_inv, 1);
  if (ok && fp8) {
    std::vector<uint8_t> q((size_t)Tk * c.H);
    std::vector<float> s((size_t)Tk * (c.H / 128));
    eplref_dispatch_fp8(T, c.k, c.H, x.data(), r_row.data(), q.data(), s.data());
    ok = same("fp8 rows", payload_rows(host_copy((const uint8_t*)d_recv, (size_t)P * PP), P, c.H, PP), q,
              (size_t)P * c.H) &&
         same("fp8 scales", host_copy(d_scale, (size_t)P * (c.H / 128)), s, (size_t)P * (c.H / 128));
  } else if (ok) {
    std::vector<uint16_t> rr((size_t)Tk * c.H);
    eplref_dispatch_bf16(T, c.k, c.H, x.data(), r_row.data(), rr.data());
    ok = same("bf16 rows", payload_rows(host_copy((const uint16_t*)d_recv, (size_t)P * PP), P, c.H, PP), rr,
              (size_t)P * c.H);
  }
  if (ok) {
    std::vector<uint16_t> o((size_t)T * c.H);
    eplref_combine(T, c.k, c.H, y.data(), w.data(), r_row.data(), nullptr, T, o.data());
    ok = same("combine", host_copy(d_o, (size_t)T * c.H), o, (size_t)T * c.H);
  }
  if (ok) {  // expert and offset of every packed row, and of one position past the end
    const int64_t n = Tk + 1;
    std::vector<int32_t> le(n), lo(n);
    eplref_locate_rows(c.E, r_eoff.data(), n, nullptr, le.data(), lo.data());
    int32_t *d_le = nullptr, *d_lo = nullptr;
    HIP_OK(hipMalloc(&d_le, n * 4));
    HIP_OK(hipMalloc(&d_lo, n * 4));
    ok = epl_locate_rows(&cfg, d_out[2], nullptr, n, d_le, d_lo, stream) == EPL_OK;
    HIP_OK(hipStreamSynchronize(stream));
    ok = ok && same("locate expert", host_copy(d_le, n), le, n) && same("locate offset", host_copy(d_lo, n), lo, n);
    HIP_OK(hipFree(d_le));
    HIP_OK(hipFree(d_lo));
  }

  if (ok && !fp8 && T > 0) {  // the hierarchical schedule and the dispatch in its order
    const int n = 6, NH = 2;
    std::vector<int32_t> hop((size_t)c.R * c.R), order(c.E);
    for (int a = 0; a < c.R; ++a)
      for (int b = 0; b < c.R; ++b) hop[(size_t)a * c.R + b] = (a / 8 == b / 8) ? 0 : 1;  // nodes of 8 ranks
    eplref_transposed_order(c.E, n, order.data());
    std::vector<int32_t> se((size_t)c.R * n), so((size_t)c.R * n), cnt((size_t)c.R * n * NH);
    eplref_hop_schedule(c.R, c.E, n, NH, r_send.data(), order.data(), hop.data(), se.data(), so.data(), cnt.data());
    int32_t* d_hop = dev_copy(hop);
    int32_t *d_se = nullptr, *d_so = nullptr, *d_cnt = nullptr;
    HIP_OK(hipMalloc(&d_se, se.size() * 4));
    HIP_OK(hipMalloc(&d_so, so.size() * 4));
    HIP_OK(hipMalloc(&d_cnt, cnt.size() * 4));
    void* d_recv2 = nullptr;
    HIP_OK(hipMalloc(&d_recv2, std::max<size_t>(1, (size_t)Tk * PP * 2)));
    ok = epl_hop_schedule(&cfg, d_out[0], nullptr, 0, d_hop, n, NH, d_se, d_so, d_cnt, stream) == EPL_OK &&
         epl_dispatch_scheduled(&cfg, d_x, &L, d_recv2, nullptr, Tk, 0, n, stream) == EPL_OK;
    HIP_OK(hipStreamSynchronize(stream));
    std::vector<uint16_t> rr((size_t)Tk * c.H);
    eplref_dispatch_bf16(T, c.k, c.H, x.data(), r_row.data(), rr.data());
    ok = ok && same("schedule start expert", host_copy(d_se, se.size()), se, se.size()) &&
         same("schedule start offset", host_copy(d_so, so.size()), so, so.size()) &&
         same("schedule class counts", host_copy(d_cnt, cnt.size()), cnt, cnt.size()) &&
         same("scheduled dispatch rows",
              payload_rows(host_copy((const uint16_t*)d_recv2, (size_t)P * PP), P, c.H, PP), rr, (size_t)P * c.H);
    ok = ok && epl_hop_schedule(&cfg, d_out[0], nullptr, 0, d_hop, 0, NH, d_se, d_so, d_cnt, stream) ==
                   EPL_ERR_INVALID_ARG &&
         epl_hop_schedule(&cfg, d_out[0], nullptr, 0, d_hop, n, EPL_MAX_HOP_CLASSES + 1, d_se, d_so, d_cnt, stream) ==
             EPL_ERR_INVALID_ARG &&
         epl_dispatch_scheduled(&cfg, d_x, &L, d_recv2, nullptr, Tk - 1, 0, n, stream) == EPL_ERR_CAPACITY &&
         epl_dispatch_scheduled(&cfg, (char*)d_x + 2, &L, d_recv2, nullptr, Tk, 0, n, stream) == EPL_ERR_ALIGN;
    HIP_OK(hipFree(d_hop));
    HIP_OK(hipFree(d_se));
    HIP_OK(hipFree(d_so));
    HIP_OK(hipFree(d_cnt));
    HIP_OK(hipFree(d_recv2));
  }

  // Host-detectable errors come back before any launch.
  if (ok) {
    epl_config bad = cfg;
    bad.num_experts = c.E + 1;
    epl_config bad_pitch = cfg;
    bad_pitch.row_pitch = c.H + 32;  // not a multiple of 64
    ok = epl_layout(&bad, d_idx, &L, ws, ws_bytes, stream) == EPL_ERR_INVALID_ARG &&
         epl_layout_dispatch(&bad_pitch, d_idx, &L, ws, ws_bytes, d_x, d_recv, d_scale, Tk, stream) ==
             EPL_ERR_INVALID_ARG &&
         epl_combine(&bad_pitch, d_y, d_w, &L, d_o, stream) == EPL_ERR_INVALID_ARG &&
         epl_layout(&cfg, d_idx, &L, ws, ws_bytes - 4, stream) == EPL_ERR_WORKSPACE &&
         epl_dispatch(&cfg, d_x, &L, d_recv, d_scale, Tk - 1, stream) == EPL_ERR_CAPACITY &&
         epl_dispatch(&cfg, d_x, &L, (char*)d_recv + 2, d_scale, Tk, stream) == EPL_ERR_ALIGN &&
         epl_layout_dispatch(&cfg, d_idx, &L, ws, ws_bytes, d_x, d_recv, d_scale, Tk - 1, stream) ==
             EPL_ERR_CAPACITY &&
         epl_layout_dispatch(&cfg, d_idx, &L, ws, ws_bytes - 4, d_x, d_recv, d_scale, Tk, stream) ==
             EPL_ERR_WORKSPACE &&
         epl_layout_counts(&cfg, d_idx, &L, ws, ws_bytes - 4, stream) == EPL_ERR_WORKSPACE &&
         epl_layout_counts(&bad, d_idx, &L, ws, ws_bytes, stream) == EPL_ERR_INVALID_ARG &&
         epl_dispatch_rows(&cfg, d_idx, &L, ws, ws_bytes, d_x, d_recv, d_scale, Tk - 1, stream) ==
             EPL_ERR_CAPACITY &&
         epl_dispatch_rows(&cfg, d_idx, &L, ws, ws_bytes, (char*)d_x + 2, d_recv, d_scale, Tk, stream) ==
             EPL_ERR_ALIGN &&
         epl_combine(&cfg, d_y, d_w, &L, (char*)d_o + 8, stream) == EPL_ERR_ALIGN;
    if (!ok) std::printf("an invalid call was not rejected with the documented status\n");
  }

  for (int32_t* p : d_out) HIP_OK(hipFree(p));
  HIP_OK(hipFree(d_idx));
  HIP_OK(hipFree(ws));
  HIP_OK(hipFree(d_x));
  HIP_OK(hipFree(d_y));
  HIP_OK(hipFree(d_w));
  HIP_OK(hipFree(d_recv));
  if (d_scale) HIP_OK(hipFree(d_scale));
  HIP_OK(hipFree(d_o));
  std::printf("case R=%d E=%d k=%d Tr=%d H=%d pitch=%d %s %s (%d launches): %s\n", c.R, c.E, c.k, c.Tr, c.H, PP,
              fp8 ? "fp8" : "bf16", kModeName[mode],
              mode == kSeparate ? epl_layout_launches(&cfg) + 1 : epl_layout_dispatch_launches(&cfg),
              ok ? "ok" : "FAILED");
  return ok;
}

// The one-launch layer synchronised by Token-Flag Fusion or Data-for-Checksum: two consecutive
// calls (epochs 1 and 2) on one marks buffer, each output against the oracle's combine of x's rows.
bool run_layer_case(int variant, uint64_t seed, hipStream_t stream) {
  const int R = 8, E = 32, k = 4, Tr = 50, H = 1024;
  const int64_t T = (int64_t)R * Tr, Tk = T * k;
  epl_config cfg{R, E, k, H, Tr, EPL_PAYLOAD_BF16, 0};
  std::vector<int32_t> idx(Tk);
  for (auto& v : idx) v = (int32_t)(splitmix(seed) % (uint64_t)(E + 2)) - 1;
  std::vector<uint16_t> x((size_t)T * H);
  for (auto& v : x) v = (uint16_t)(0x3C00 + (splitmix(seed) % 0x0800) - 0x0400);
  std::vector<float> w(Tk);
  for (auto& v : w) v = (float)(splitmix(seed) % 1000) / 1000.0f;
  std::vector<int32_t> r_send(R * E), r_rank(R * R), r_eoff(E + 1), r_roff(R + 1), r_seg(E * R), r_ntok(T), r_row(Tk),
      r_slot(Tk), r_src(Tk), r_j(Tk), r_inv(1);
  eplref_layout(R, E, k, Tr, idx.data(), r_send.data(), r_rank.data(), r_eoff.data(), r_roff.data(), r_seg.data(),
                r_ntok.data(), r_row.data(), r_slot.data(), r_src.data(), r_j.data(), r_inv.data());
  const int32_t P = r_eoff[E];
  std::vector<uint16_t> y((size_t)std::max<int32_t>(P, 1) * H);
  for (int32_t r = 0; r < P; ++r) std::memcpy(&y[(size_t)r * H], &x[(size_t)r_src[r] * H], H * 2);
  std::vector<uint16_t> want((size_t)T * H);
  eplref_combine(T, k, H, y.data(), w.data(), r_row.data(), nullptr, T, want.data());

  int32_t* d_idx = dev_copy(idx);
  const size_t sizes[] = {(size_t)R * E, (size_t)R * R, (size_t)E + 1, (size_t)R + 1, (size_t)E * R, (size_t)T,
                          (size_t)Tk,    (size_t)Tk,    (size_t)Tk,    (size_t)Tk,    1};
  std::vector<int32_t*> d_out;
  for (size_t n : sizes) {
    int32_t* q = nullptr;
    HIP_OK(hipMalloc(&q, n * 4));
    d_out.push_back(q);
  }
  epl_layout_buffers L{d_out[0], d_out[1], d_out[2], d_out[3], d_out[4], d_out[5],
                       d_out[6], d_out[7], d_out[8], d_out[9], d_out[10]};
  const size_t ws_bytes = epl_workspace_bytes(&cfg);
  void* ws = nullptr;
  HIP_OK(hipMalloc(&ws, ws_bytes));
  HIP_OK(hipMemset(ws, 0, ws_bytes));  // the one-launch calls' synchronisation words start at zero
  uint16_t* d_x = dev_copy(x);
  float* d_w = dev_copy(w);
  void *d_recv = nullptr, *d_o = nullptr, *d_marks = nullptr;
  int32_t* d_status = nullptr;
  HIP_OK(hipMalloc(&d_recv, (size_t)Tk * H * 2));
  HIP_OK(hipMalloc(&d_o, (size_t)T * H * 2));
  const int64_t marks_bytes = epl_layer_marks_bytes(&cfg, Tk);
  HIP_OK(hipMalloc(&d_marks, marks_bytes));
  HIP_OK(hipMemset(d_marks, 0, marks_bytes));
  HIP_OK(hipMalloc(&d_status, 4));
  bool ok = marks_bytes == Tk * 2 * 8;
  for (uint64_t epoch = 1; ok && epoch <= 2; ++epoch) {
    ok = epl_layer_data_as_flag(&cfg, d_idx, &L, ws, ws_bytes, d_x, d_recv, Tk, d_w, d_o, (uint64_t*)d_marks,
                                variant, epoch, nullptr, d_status, stream) == EPL_OK;
    HIP_OK(hipStreamSynchronize(stream));
    ok = ok && host_copy(d_status, 1)[0] == 0 && same("layer pair_row", host_copy(d_out[6], Tk), r_row, Tk) &&
         same("layer combine", host_copy((const uint16_t*)d_o, (size_t)T * H), want, (size_t)T * H);
  }
  ok = ok &&
       epl_layer_data_as_flag(&cfg, d_idx, &L, ws, ws_bytes, d_x, d_recv, Tk, d_w, d_o, (uint64_t*)d_marks, variant,
                              0, nullptr, d_status, stream) == EPL_ERR_INVALID_ARG &&
       epl_layer_data_as_flag(&cfg, d_idx, &L, ws, ws_bytes, d_x, d_recv, Tk, d_w, d_o, (uint64_t*)d_marks, 7, 3,
                              nullptr, d_status, stream) == EPL_ERR_INVALID_ARG &&
       epl_layer_data_as_flag(&cfg, d_idx, &L, ws, ws_bytes, d_x, d_recv, Tk, d_w, d_o,
                              (uint64_t*)((char*)d_marks + 4), variant, 3, nullptr, d_status,
                              stream) == EPL_ERR_ALIGN;
  for (int32_t* q : d_out) HIP_OK(hipFree(q));
  HIP_OK(hipFree(d_idx));
  HIP_OK(hipFree(ws));
  HIP_OK(hipFree(d_x));
  HIP_OK(hipFree(d_w));
  HIP_OK(hipFree(d_recv));
  HIP_OK(hipFree(d_o));
  HIP_OK(hipFree(d_marks));
  HIP_OK(hipFree(d_status));
  std::printf("layer R=%d E=%d k=%d Tr=%d H=%d %s, epochs 1 and 2: %s\n", R, E, k, Tr, H,
              variant == EPL_DAF_TOKEN_FLAG_FUSION ? "Token-Flag Fusion" : "Data-for-Checksum", ok ? "ok" : "FAILED");
  return ok;
}

}  // namespace

int main() {
  std::printf("%s\n", epl_version());
  hipStream_t stream;
  HIP_OK(hipStreamCreate(&stream));
  const Case cases[] = {
      {8, 32, 4, 50, 1024, EPL_PAYLOAD_BF16},     // one-launch layout
      {4, 16, 8, 100, 512, EPL_PAYLOAD_FP8_E4M3},  // fp8, one-launch layout
      {32, 256, 8, 80, 256, EPL_PAYLOAD_BF16},    // T*k = 20480: three-launch layout
      {64, 256, 8, 40, 1024, EPL_PAYLOAD_BF16},   // finalize fused into the row kernel
      {2, 8, 3, 0, 64, EPL_PAYLOAD_BF16},         // no tokens
      {64, 256, 8, 40, 1024, EPL_PAYLOAD_BF16, 1024 + 768},  // fused, rows 1.5 KiB apart beyond their 2 KiB
      {4, 16, 8, 100, 512, EPL_PAYLOAD_FP8_E4M3, 576},       // fp8 rows 64 bytes apart beyond their 512
      {32, 256, 8, 80, 256, EPL_PAYLOAD_BF16, 320},          // three-launch layout, padded rows
  };
  bool ok = true;
  uint64_t seed = 12345;
  for (const Case& c : cases) {
    for (Mode m : {kSeparate, kOneCall, kTwoPhases}) ok = run_case(c, seed, stream, m) && ok;
    ++seed;
  }
  for (int variant : {EPL_DAF_TOKEN_FLAG_FUSION, EPL_DAF_DATA_CHECKSUM}) ok = run_layer_case(variant, seed++, stream) && ok;
  HIP_OK(hipStreamDestroy(stream));
  if (!ok) return 1;
  std::printf("c abi check ok\n");
  return 0;
}
