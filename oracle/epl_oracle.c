/*
 * CPU oracle for MoE token dispatch / combine -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, single-threaded C99. Only the tests, the smoke check and the benchmark's CPU
 * baseline call it; the product path never does. It shares no code, header, table or helper
 * with the GPU library.
 *
 * What it computes. The paper's dispatch routes every (token, chosen expert) pair to the rank
 * hosting that expert. The receive space is split by (source rank, expert) from per-expert token
 * counts; the receiver then turns the counts into prefix-sum offsets and reorders tokens
 * contiguously per expert (Background, "Deploying MoE on CM384", phases 1-5; Kernel
 * Decomposition: CalCumSum gives per-expert HBM offsets). Combine gathers expert outputs back
 * into token order (Background; Overview says combine is not elaborated). Here the final packed
 * layout is written out directly as a stable counting sort of the valid pairs by expert id. Rows
 * therefore run in (destination rank, expert, source rank, token, j) order.
 *
 * Notation: R ranks, E experts (E % R == 0, El = E/R per rank, rank of expert e is e/El),
 * k = top-k, Tr tokens per rank, T = R*Tr tokens, H hidden size. Pair p = g*k + j of token g
 * is valid iff 0 <= idx[p] < E. The source rank of token g is g/Tr.
 *
 * Readings where the paper is silent are these:
 *  - invalid ids are skipped and counted;
 *  - duplicate ids in one token are separate pairs;
 *  - dedup is metadata only;
 *  - combine applies the weights as given, as an fp32 fmaf chain in j order from +0, then bf16 RNE;
 *  - fp8 is OCP E4M3 (max 448) with one fp32 scale amax/448 per 128-element block.
 *
 * Every function is pinned by the non-GPU tests, against brute force, closed forms, invariants
 * and library routines.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define REF_API __attribute__((visibility("default")))

static int ref_valid(int32_t e, int E) { return e >= 0 && e < E; }

/* ------------------------------------------------------------------------------------------
 * Layout: counts, offsets, slots, dedup. Returns 0 on success, -1 on a bad shape.
 *   send_cnt  [R*E]  pairs of source rank s routed to expert e           (per-expert token counts)
 *   rank_cnt  [R*R]  tokens of source rank s whose destination set contains rank r
 *   expert_off[E+1]  exclusive prefix sum over e of sum_s send_cnt[s][e] (CalCumSum offsets)
 *   rank_off  [R+1]  expert_off[d*El]
 *   seg_off   [E*R]  seg_off[e*R+s] = expert_off[e] + sum_{s'<s} send_cnt[s'][e]
 *   tok_nranks[T]    number of distinct destination ranks of token g
 *   pair_row  [T*k]  packed receive row of pair p, -1 if invalid
 *   pair_rslot[T*k]  slot of token g among tokens of its rank bound for rank(idx[p]), -1 invalid
 *   recv_src  [T*k]  recv_src[row] = g for rows < P (rest untouched)
 *   recv_j    [T*k]  recv_j[row] = j
 *   num_invalid[1]
 * ------------------------------------------------------------------------------------------ */
REF_API int eplref_layout(int R, int E, int k, int Tr, const int32_t *idx, int32_t *send_cnt,
                          int32_t *rank_cnt, int32_t *expert_off, int32_t *rank_off, int32_t *seg_off,
                          int32_t *tok_nranks, int32_t *pair_row, int32_t *pair_rslot, int32_t *recv_src,
                          int32_t *recv_j, int32_t *num_invalid) {
  if (R < 1 || E < R || E % R != 0 || k < 1 || Tr < 0) return -1;
  const int El = E / R;
  const int64_t T = (int64_t)R * Tr;

  /* O1: per-(source rank, expert) counts and the invalid count. */
  memset(send_cnt, 0, sizeof(int32_t) * (size_t)R * E);
  int32_t invalid = 0;
  for (int64_t g = 0; g < T; ++g) {
    const int s = (int)(g / Tr);
    for (int j = 0; j < k; ++j) {
      const int32_t e = idx[g * k + j];
      if (ref_valid(e, E))
        send_cnt[(int64_t)s * E + e] += 1;
      else
        invalid += 1;
    }
  }
  *num_invalid = invalid;

  /* O2: per-expert totals, then exclusive prefix sums (CalCumSum). */
  expert_off[0] = 0;
  for (int e = 0; e < E; ++e) {
    int32_t recv = 0;
    for (int s = 0; s < R; ++s) recv += send_cnt[(int64_t)s * E + e];
    expert_off[e + 1] = expert_off[e] + recv;
  }
  for (int d = 0; d <= R; ++d) rank_off[d] = expert_off[d * El];

  /* O3: each expert's segment is split by source rank, ranks ascending. */
  for (int e = 0; e < E; ++e) {
    int32_t off = expert_off[e];
    for (int s = 0; s < R; ++s) {
      seg_off[(int64_t)e * R + s] = off;
      off += send_cnt[(int64_t)s * E + e];
    }
  }

  /* O4/O5: counting-sort placement. A cursor per (expert, source) segment, advanced in pair
   * order, gives each pair its stable slot in that segment. */
  int32_t *cursor = (int32_t *)malloc(sizeof(int32_t) * ((size_t)R * E + 1));
  if (!cursor) return -1;
  memcpy(cursor, seg_off, sizeof(int32_t) * (size_t)R * E);
  for (int64_t g = 0; g < T; ++g) {
    const int s = (int)(g / Tr);
    for (int j = 0; j < k; ++j) {
      const int64_t p = g * k + j;
      const int32_t e = idx[p];
      if (!ref_valid(e, E)) {
        pair_row[p] = -1;
        continue;
      }
      const int32_t row = cursor[(int64_t)e * R + s]++;
      pair_row[p] = row;
      recv_src[row] = (int32_t)g;
      recv_j[row] = j;
    }
  }
  free(cursor);

  /* O6: destination-rank dedup. A pair is the first of its token for a rank if no earlier
   * valid pair of the same token goes to that rank. Each such (token, rank) takes the next
   * slot among its source rank's tokens bound for that rank; every pair of the token on that
   * rank reports the same slot. */
  memset(rank_cnt, 0, sizeof(int32_t) * (size_t)R * R);
  for (int64_t g = 0; g < T; ++g) {
    const int s = (int)(g / Tr);
    int32_t nranks = 0;
    for (int j = 0; j < k; ++j) {
      const int64_t p = g * k + j;
      const int32_t e = idx[p];
      if (!ref_valid(e, E)) {
        pair_rslot[p] = -1;
        continue;
      }
      const int d = e / El;
      int first_j = -1;
      for (int jj = 0; jj < j; ++jj) {
        const int32_t e2 = idx[g * k + jj];
        if (ref_valid(e2, E) && e2 / El == d) {
          first_j = jj;
          break;
        }
      }
      if (first_j < 0) {
        pair_rslot[p] = rank_cnt[(int64_t)s * R + d]++;
        nranks += 1;
      } else {
        pair_rslot[p] = pair_rslot[g * k + first_j];
      }
    }
    tok_nranks[g] = nranks;
  }
  return 0;
}

/* ------------------------------------------------------------------------------------------
 * Number formats, written from their definitions.
 * ------------------------------------------------------------------------------------------ */
REF_API float eplref_bf16_to_f32(uint16_t h) {
  uint32_t u = (uint32_t)h << 16; /* bf16 is the upper half of an IEEE binary32 */
  float f;
  memcpy(&f, &u, 4);
  return f;
}

/* Nearest bf16 value to v, ties to the value with an even last mantissa bit. bf16 has 8
 * significant bits: in the binade [2^b, 2^(b+1)) its spacing is 2^(b-7); below 2^-126 the
 * spacing is 2^-133. Magnitudes that round to 2^128 or beyond become infinity. */
REF_API uint16_t eplref_f32_to_bf16(float v) {
  uint32_t u;
  memcpy(&u, &v, 4);
  if (isnan(v)) return (uint16_t)((u >> 16) | 0x0040u);
  const double a = fabs((double)v);
  double r;
  if (isinf(v) || a == 0.0) {
    r = a;
  } else {
    int ex;
    frexp(a, &ex); /* a = f * 2^ex, f in [0.5, 1) -> binade 2^(ex-1) */
    int b = ex - 1;
    if (b < -126) b = -126;
    const double q = ldexp(1.0, b - 7);
    r = nearbyint(a / q) * q; /* a / q is exact; nearbyint rounds half to even */
    if (r >= ldexp(1.0, 128)) r = INFINITY;
  }
  const float rf = (float)(signbit(v) ? -r : r); /* exact: r is on the bf16 grid */
  uint32_t ru;
  memcpy(&ru, &rf, 4);
  return (uint16_t)(ru >> 16);
}

/* OCP 8-bit floating point, E4M3 ("fn"): bias 7, no infinities, S.1111.111 is NaN, largest
 * finite magnitude 448 (S.1111.110), smallest normal 2^-6, subnormal spacing 2^-9. */
REF_API float eplref_e4m3_to_f32(uint8_t c) {
  const int sign = c >> 7, ex = (c >> 3) & 15, man = c & 7;
  double v;
  if (ex == 15 && man == 7)
    v = NAN;
  else if (ex == 0)
    v = ldexp((double)man, -9);
  else
    v = ldexp(8.0 + man, ex - 7 - 3);
  return (float)(sign ? -v : v);
}

/* Round to the nearest E4M3 value, ties to an even mantissa, saturating magnitudes >= 448 to
 * 448 and keeping the sign of values that round to zero. */
REF_API uint8_t eplref_f32_to_e4m3(float v) {
  const uint8_t sign = signbit(v) ? 0x80 : 0x00;
  if (isnan(v)) return (uint8_t)(sign | 0x7F);
  const double a = fabs((double)v);
  if (a >= 448.0) return (uint8_t)(sign | 0x7E);
  int b = -6; /* binade exponent; subnormals share the spacing of the lowest normal binade */
  if (a >= ldexp(1.0, -6)) {
    int ex;
    frexp(a, &ex);
    b = ex - 1;
  }
  const double q = ldexp(1.0, b - 3);
  const double r = nearbyint(a / q) * q; /* rounded magnitude; never above 448 here */
  if (r == 0.0) return sign;
  if (r < ldexp(1.0, -6)) return (uint8_t)(sign | (uint8_t)(r / ldexp(1.0, -9)));
  int ex;
  frexp(r, &ex);
  const int field = (ex - 1) + 7;
  const int man = (int)(r / ldexp(1.0, ex - 1) * 8.0) - 8;
  return (uint8_t)(sign | (field << 3) | man);
}

REF_API void eplref_f32_to_bf16_array(const float *in, uint16_t *out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = eplref_f32_to_bf16(in[i]);
}
REF_API void eplref_f32_to_e4m3_array(const float *in, uint8_t *out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = eplref_f32_to_e4m3(in[i]);
}

/* ------------------------------------------------------------------------------------------
 * Dispatch. Every valid pair's token row is written to its packed receive row.
 * ------------------------------------------------------------------------------------------ */
REF_API void eplref_dispatch_bf16(int64_t T, int k, int H, const uint16_t *x, const int32_t *pair_row,
                                  uint16_t *recv) {
  for (int64_t g = 0; g < T; ++g)
    for (int j = 0; j < k; ++j) {
      const int32_t row = pair_row[g * k + j];
      if (row >= 0) memcpy(recv + (int64_t)row * H, x + g * H, sizeof(uint16_t) * (size_t)H);
    }
}

/* FP8 quantisation of one token row: per 128-element block b, a = max |x|, s = a / 448
 * (fp32 division), q = E4M3(x / s) (fp32 division); a block with a == 0 has s = 0, q = 0. */
REF_API void eplref_quantize_row_e4m3(int H, const uint16_t *xrow, uint8_t *q, float *scale) {
  for (int b = 0; b < H / 128; ++b) {
    float a = 0.0f;
    for (int c = 0; c < 128; ++c) {
      const float m = fabsf(eplref_bf16_to_f32(xrow[b * 128 + c]));
      if (m > a) a = m;
    }
    const float s = a / 448.0f;
    scale[b] = s;
    for (int c = 0; c < 128; ++c)
      q[b * 128 + c] = (a == 0.0f) ? 0 : eplref_f32_to_e4m3(eplref_bf16_to_f32(xrow[b * 128 + c]) / s);
  }
}

REF_API void eplref_dispatch_fp8(int64_t T, int k, int H, const uint16_t *x, const int32_t *pair_row,
                                 uint8_t *recv, float *recv_scale) {
  const int NB = H / 128;
  uint8_t *q = (uint8_t *)malloc((size_t)H);
  float *sc = (float *)malloc(sizeof(float) * (size_t)(NB > 0 ? NB : 1));
  for (int64_t g = 0; g < T; ++g) {
    eplref_quantize_row_e4m3(H, x + g * H, q, sc);
    for (int j = 0; j < k; ++j) {
      const int32_t row = pair_row[g * k + j];
      if (row < 0) continue;
      memcpy(recv + (int64_t)row * H, q, (size_t)H);
      memcpy(recv_scale + (int64_t)row * NB, sc, sizeof(float) * (size_t)NB);
    }
  }
  free(q);
  free(sc);
}

/* ------------------------------------------------------------------------------------------
 * Combine: out[g][c] = BF16( fold over j = 0..k-1 with pair_row >= 0 of
 *                            acc = fmaf(w[g][j], float(y[pair_row][c]), acc) ), acc starts at +0.
 * tokens == NULL combines every token 0..T-1 into out[g]; otherwise it combines the listed
 * tokens, writing token tokens[i] to out row i.
 * ------------------------------------------------------------------------------------------ */
REF_API void eplref_combine(int64_t T, int k, int H, const uint16_t *y, const float *w,
                            const int32_t *pair_row, const int64_t *tokens, int64_t n_tokens, uint16_t *out) {
  const int64_t n = tokens ? n_tokens : T;
  for (int64_t i = 0; i < n; ++i) {
    const int64_t g = tokens ? tokens[i] : i;
    for (int c = 0; c < H; ++c) {
      float acc = 0.0f;
      for (int j = 0; j < k; ++j) {
        const int32_t row = pair_row[g * k + j];
        if (row < 0) continue;
        acc = fmaf(w[g * k + j], eplref_bf16_to_f32(y[(int64_t)row * H + c]), acc);
      }
      out[i * H + c] = eplref_f32_to_bf16(acc);
    }
  }
}

/* Same as eplref_combine, but y rows are looked up through a row map: expert row `row` is
 * found at ys[row_map[row]]. Used when only a sample of y has been copied to the host. */
REF_API void eplref_combine_mapped(int k, int H, const uint16_t *ys, const int32_t *row_map, const float *w,
                                   const int32_t *pair_row, const int64_t *tokens, int64_t n_tokens,
                                   uint16_t *out) {
  for (int64_t i = 0; i < n_tokens; ++i) {
    const int64_t g = tokens[i];
    for (int c = 0; c < H; ++c) {
      float acc = 0.0f;
      for (int j = 0; j < k; ++j) {
        const int32_t row = pair_row[g * k + j];
        if (row < 0) continue;
        acc = fmaf(w[g * k + j], eplref_bf16_to_f32(ys[(int64_t)row_map[row] * H + c]), acc);
      }
      out[i * H + c] = eplref_f32_to_bf16(acc);
    }
  }
}

/* ------------------------------------------------------------------------------------------
 * Row location (Hierarchical Token-level Scheduling, Token-level Load Partition; Algorithm 1):
 * a global position in the expert-major packed rows is mapped to the expert whose cumulative
 * range covers it and the position's offset inside that expert's rows. The plain definition
 * is written out as a linear scan: expert e with expert_off[e] <= r < expert_off[e+1] (the
 * unique non-empty such e), offset r - expert_off[e]. rows == NULL means r = i for i = 0..n-1.
 * Positions outside [0, expert_off[E]) get expert -1 and offset -1.
 * ------------------------------------------------------------------------------------------ */
REF_API void eplref_locate_rows(int E, const int32_t *expert_off, int64_t n, const int32_t *rows, int32_t *expert,
                                int32_t *offset) {
  const int64_t P = expert_off[E];
  for (int64_t i = 0; i < n; ++i) {
    const int64_t r = rows ? rows[i] : i;
    expert[i] = -1;
    offset[i] = -1;
    if (r < 0 || r >= P) continue;
    for (int e = 0; e < E; ++e)
      if (expert_off[e] <= r && r < expert_off[e + 1]) {
        expert[i] = e;
        offset[i] = (int32_t)(r - expert_off[e]);
        break;
      }
  }
}

/* ------------------------------------------------------------------------------------------
 * Hierarchical token-level scheduling (Hierarchical Token-level Scheduling: latency
 * homogenization, the hardware-accelerated mapper's expert remapping by logical matrix
 * transposition and token-level load partition).
 *
 * The remapped expert sequence, as the reading of the transposition: a virtual matrix of `rows`
 * rows (the paper: one row per worker) and c = ceil(E/rows) columns holds the experts in their
 * natural order, row by row (row w holds experts w*c .. w*c+c-1, the block a worker would take
 * without the remap); the sequence reads it column by column, skipping the cells past E.
 * ------------------------------------------------------------------------------------------ */
REF_API void eplref_transposed_order(int E, int rows, int32_t *order) {
  const int c = (E + rows - 1) / rows;
  int i = 0;
  for (int col = 0; col < c; ++col)
    for (int row = 0; row < rows; ++row) {
      const int e = row * c + col;
      if (e < E) order[i++] = e;
    }
}

/* For each source rank s: the pairs it sends, taken expert by expert in the sequence `order`
 * (order[i] is the i-th expert; it contributes send_cnt[s][order[i]] pairs), are cut into n
 * contiguous slices whose sizes differ by at most one: slice j is positions
 * [floor(j*m/n), floor((j+1)*m/n)) of the m pairs. Worker j of source s gets
 *   start_expert[s*n+j], start_offset[s*n+j]: the expert of the slice's first position and that
 *       position's offset among the expert's pairs (-1, -1 for an empty slice);
 *   counts[(s*n+j)*NH+h]: the slice's pairs whose destination rank d = e / (E/R) has hop class
 *       hop[s*R+d] == h, for 0 <= h < NH (a class outside that range is counted nowhere).
 * Written as the plain definition: the overlap of every expert's range with the slice. */
REF_API void eplref_hop_schedule(int R, int E, int n, int NH, const int32_t *send_cnt, const int32_t *order,
                                 const int32_t *hop, int32_t *start_expert, int32_t *start_offset,
                                 int32_t *counts) {
  const int El = E / R;
  for (int s = 0; s < R; ++s) {
    int64_t m = 0;
    for (int e = 0; e < E; ++e) m += send_cnt[(int64_t)s * E + e];
    for (int j = 0; j < n; ++j) {
      const int64_t lo = (int64_t)j * m / n, hi = (int64_t)(j + 1) * m / n;
      int32_t *cnt = counts + ((int64_t)s * n + j) * NH;
      for (int h = 0; h < NH; ++h) cnt[h] = 0;
      start_expert[(int64_t)s * n + j] = -1;
      start_offset[(int64_t)s * n + j] = -1;
      int64_t base = 0;
      for (int i = 0; i < E; ++i) {
        const int e = order[i];
        const int64_t c = send_cnt[(int64_t)s * E + e];
        const int64_t a = base > lo ? base : lo;
        const int64_t b = base + c < hi ? base + c : hi;
        if (b > a) {
          const int32_t h = hop[(int64_t)s * R + e / El];
          if (h >= 0 && h < NH) cnt[h] += (int32_t)(b - a);
          if (start_expert[(int64_t)s * n + j] < 0) {
            start_expert[(int64_t)s * n + j] = e;
            start_offset[(int64_t)s * n + j] = (int32_t)(lo - base);
          }
        }
        base += c;
      }
    }
  }
}
