/*
 * moe_oracle.c -- plain, slow, obviously-correct CPU oracle for one
 * expert-parallel rank's MoE expert stage.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
 * load this file; only the tests, the smoke check and the benchmark's CPU
 * baseline leg use it.  It shares no code, header or table with the HIP
 * library.
 *
 * What it computes (paper Section 2.1, steps 3-4: each rank runs the expert
 * computation of its local experts on the routed token copies it received,
 * and each expert output row returns to the rank the token came from, into
 * the slot that rank reserved for it).  The expert is the SiLU-gated FFN
 *     y = W2_e * bf16( silu(W1_e x) (.) (W3_e x) ),   silu(g) = g / (1 + e^-g),
 * and for every routed row i of local expert e:
 *     return_bufs[src[i]][slot[i], :] = bf16_rne(y_i).
 * Nothing else in the return buffers is written.  moe_oracle_combine adds the
 * step after (Section 2.1, step 5): each source rank's gate-weighted sum of
 * its tokens' returned rows.  The row layout, tile
 * schedule, segments and overlap of the paper's method (Section 3) change
 * only when and where rows are computed, never their values, so the oracle
 * has none of them.
 *
 * Precision: inputs are bf16; products of two bf16 values are exact in fp32
 * and every dot product accumulates in fp32 in ascending index order.  The
 * gated activation is rounded to bf16 exactly once (the down projection
 * consumes bf16 operands), and the output is rounded to bf16 (RNE).
 *
 * Validation (same codes as the library): -1 invalid argument, -2 bad
 * routing (offsets not monotone from 0 to rows, source rank out of range,
 * slot outside its receive buffer, or two rows with the same (rank, slot)).
 *
 * Compile-time ORACLE_MUTATION (default 0) plants a deliberate mistake; it
 * exists only so the tests can show that the oracle's pins catch it.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#ifndef ORACLE_MUTATION
#define ORACLE_MUTATION 0
#endif

enum { OR_OK = 0, OR_EINVAL = -1, OR_EROUTING = -2 };

static float widen_bf16(uint16_t v) {
  uint32_t u = (uint32_t)v << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

static uint16_t round_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u); /* quiet NaN */
  u += 0x7fffu + ((u >> 16) & 1u);                                           /* nearest-even */
  return (uint16_t)(u >> 16);
}

/* Checks the routing arguments; returns 0 or a negative code. */
int moe_oracle_validate(int32_t hidden, int32_t ffn, int32_t num_local_experts, int32_t num_ranks,
                        int32_t self_rank, int64_t rows, const int32_t* expert_offsets,
                        const int32_t* row_src_rank, const int32_t* row_slot,
                        const int64_t* return_rows) {
  if (hidden <= 0 || ffn <= 0 || num_local_experts <= 0 || num_ranks <= 0) return OR_EINVAL;
  if (self_rank < 0 || self_rank >= num_ranks || rows < 0) return OR_EINVAL;
  if (!expert_offsets || !return_rows) return OR_EINVAL;
  if (rows > 0 && (!row_src_rank || !row_slot)) return OR_EINVAL;
  for (int r = 0; r < num_ranks; ++r)
    if (return_rows[r] < 0) return OR_EINVAL;

  if (expert_offsets[0] != 0 || expert_offsets[num_local_experts] != rows) return OR_EROUTING;
  for (int e = 0; e < num_local_experts; ++e)
    if (expert_offsets[e] > expert_offsets[e + 1]) return OR_EROUTING;

  /* One byte per receive-buffer row marks slots already claimed. */
  unsigned char** seen = (unsigned char**)calloc((size_t)num_ranks, sizeof(unsigned char*));
  if (!seen) return OR_EINVAL;
  int rc = OR_OK;
  for (int r = 0; r < num_ranks && rc == OR_OK; ++r) {
    seen[r] = (unsigned char*)calloc((size_t)return_rows[r] + 1, 1);
    if (!seen[r]) rc = OR_EINVAL;
  }
  for (int64_t i = 0; i < rows && rc == OR_OK; ++i) {
    int32_t r = row_src_rank[i];
    if (r < 0 || r >= num_ranks) { rc = OR_EROUTING; break; }
    int32_t s = row_slot[i];
    if (s < 0 || (int64_t)s >= return_rows[r]) { rc = OR_EROUTING; break; }
    if (seen[r][s]) { rc = OR_EROUTING; break; }
    seen[r][s] = 1;
  }
  for (int r = 0; r < num_ranks; ++r) free(seen[r]);
  free(seen);
  return rc;
}

/*
 * Runs the stage.  All pointers are host pointers:
 *   x            [rows, hidden] bf16, expert-contiguous (rows of local expert e are
 *                expert_offsets[e] .. expert_offsets[e+1]-1)
 *   w1, w3       [E_l, ffn, hidden] bf16 (row f holds the weights of output feature f)
 *   w2           [E_l, hidden, ffn] bf16
 *   return_bufs  array of num_ranks pointers, buffer r is [return_rows[r], hidden] bf16
 * num_threads <= 0 uses the OpenMP default.  Returns 0 or a negative code; on
 * error nothing is written.
 */
int moe_oracle_run(int32_t hidden, int32_t ffn, int32_t num_local_experts, int32_t num_ranks,
                   int32_t self_rank, int64_t rows, const uint16_t* x,
                   const int32_t* expert_offsets, const int32_t* row_src_rank,
                   const int32_t* row_slot, const uint16_t* w1, const uint16_t* w3,
                   const uint16_t* w2, uint16_t* const* return_bufs,
                   const int64_t* return_rows, int32_t num_threads) {
  int rc = moe_oracle_validate(hidden, ffn, num_local_experts, num_ranks, self_rank, rows,
                               expert_offsets, row_src_rank, row_slot, return_rows);
  if (rc != OR_OK) return rc;
  if (rows == 0) return OR_OK;
  if (!x || !w1 || !w3 || !w2 || !return_bufs) return OR_EINVAL;
  for (int r = 0; r < num_ranks; ++r)
    if (!return_bufs[r] && return_rows[r] > 0) return OR_EINVAL;

  const int64_t H = hidden, F = ffn;
  int32_t* row_expert = (int32_t*)malloc((size_t)rows * sizeof(int32_t));
  if (!row_expert) return OR_EINVAL;
  for (int e = 0; e < num_local_experts; ++e)
    for (int64_t i = expert_offsets[e]; i < expert_offsets[e + 1]; ++i) row_expert[i] = e;

#ifdef _OPENMP
  if (num_threads > 0) omp_set_num_threads(num_threads);
#else
  (void)num_threads;
#endif

#pragma omp parallel
  {
    float* xf = (float*)malloc((size_t)H * sizeof(float));
    float* a = (float*)malloc((size_t)F * sizeof(float));
#pragma omp for schedule(dynamic, 1)
    for (int64_t i = 0; i < rows; ++i) {
      const int64_t e = row_expert[i];
      const uint16_t* xi = x + i * H;
      const uint16_t* W1 = w1 + e * F * H;
      const uint16_t* W3 = w3 + e * F * H;
      const uint16_t* W2 = w2 + e * H * F;
#if ORACLE_MUTATION == 4
      W2 = w2 + ((e + 1) % num_local_experts) * H * F; /* planted: wrong expert's W2 */
#endif
      for (int64_t h = 0; h < H; ++h) xf[h] = widen_bf16(xi[h]);

      /* Gate and up projections, then the SiLU-gated product rounded once to bf16. */
      for (int64_t f = 0; f < F; ++f) {
        float g = 0.0f, u = 0.0f;
        for (int64_t h = 0; h < H; ++h) {
          g += xf[h] * widen_bf16(W1[f * H + h]);
          u += xf[h] * widen_bf16(W3[f * H + h]);
        }
#if ORACLE_MUTATION == 1
        u = 1.0f; /* planted: dropped up projection */
#endif
        float silu = g / (1.0f + expf(-g));
#if ORACLE_MUTATION == 2
        silu = g / (1.0f + expf(g)); /* planted: wrong sign inside the sigmoid */
#endif
        a[f] = widen_bf16(round_bf16(silu * u));
      }

      /* Down projection; the result goes to the slot its source rank reserved. */
      uint16_t* out = return_bufs[row_src_rank[i]] + (int64_t)row_slot[i] * H;
#if ORACLE_MUTATION == 5
      out = return_bufs[row_src_rank[i]] +
            ((int64_t)row_slot[i] + 1) % return_rows[row_src_rank[i]] * H; /* planted: wrong slot */
#endif
      for (int64_t o = 0; o < H; ++o) {
        float y = 0.0f;
        for (int64_t f = 0; f < F; ++f) {
#if ORACLE_MUTATION == 3
          y += a[f] * widen_bf16(W2[f * H + o]); /* planted: W2 read as if stored [ffn, hidden] */
#else
          y += a[f] * widen_bf16(W2[o * F + f]);
#endif
        }
        out[o] = round_bf16(y);
      }
    }
    free(xf);
    free(a);
  }
  free(row_expert);
  return OR_OK;
}

/*
 * Weighted combine on a source rank (paper Section 2.1, step 5: once the expert outputs are
 * back, each rank reduces the k outputs of every token it sent, weighted by the router's gate
 * values).  For token t of this rank:
 *     out[t, :] = bf16_rne( sum_{j = 0..k-1} gate[t*k + j] * recv[slot[t*k + j], :] ),
 * the sum in fp32 over j ascending, each term an fp32 product followed by an fp32 add (built
 * without contraction).  recv is the rank's receive buffer [recv_rows, H] bf16.
 * Returns -1 for bad sizes or null pointers, -2 if a slot is outside [0, recv_rows); then
 * nothing is written.
 */
int moe_oracle_combine(int32_t hidden, int32_t k, int64_t tokens, int64_t recv_rows, const uint16_t* recv,
                       const int32_t* slot, const float* gate, uint16_t* out, int32_t nthreads) {
  if (hidden <= 0 || k <= 0 || tokens < 0 || recv_rows < 0) return OR_EINVAL;
  if (tokens > 0 && (!recv || !slot || !gate || !out)) return OR_EINVAL;
  for (int64_t i = 0; i < tokens * k; ++i)
    if (slot[i] < 0 || slot[i] >= recv_rows) return OR_EROUTING;
  const int64_t H = hidden;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(static)
#endif
  for (int64_t t = 0; t < tokens; ++t) {
    for (int64_t h = 0; h < H; ++h) {
      float acc = 0.0f;
      for (int32_t j = 0; j < k; ++j) {
#if ORACLE_MUTATION == 7
        const int32_t s = slot[t * k];  /* planted: every term reads the first choice's row */
#else
        const int32_t s = slot[t * k + j];
#endif
#if ORACLE_MUTATION == 6
        const float term = widen_bf16(recv[s * H + h]);  /* planted: gate weight dropped */
#else
        const float term = gate[t * k + j] * widen_bf16(recv[s * H + h]);
#endif
        acc = acc + term;
      }
      out[t * H + h] = round_bf16(acc);
    }
  }
  return OR_OK;
}
