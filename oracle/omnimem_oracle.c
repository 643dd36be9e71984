/*
 * omnimem_oracle.c -- plain, slow, fp64 CPU oracle for OmniMem's memory-retrieval
 * attention step (arXiv 2605.30519).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library calls, links or loads
 * this file; only the test-suite, the smoke check and the CPU-baseline leg of the
 * benchmark do.  It shares no code, header, table or helper with the GPU path.
 *
 * Every quantity is computed in double precision on the exact input values
 * (fp32 or bf16 inputs are widened exactly), with no blocking, fusion or
 * reordering beyond what the definitions state, so each function can be checked
 * against the paper by eye.  OpenMP only distributes independent outputs over
 * threads; the arithmetic of each output is sequential and deterministic.
 *
 * Data model (the paper's notation, App. A and App. C):
 *   H heads, head dimension d, S tokens per chunk, n cached history chunks,
 *   B tokens per KV block, Bpc = ceil(S/B) blocks per chunk (chunk-aligned
 *   blocks: the last block of a chunk holds S-(Bpc-1)*B tokens).
 *   Q  : [Lq][H][d]      queries of the current chunk
 *   K,V: [n][S][H][d]    the full-resolution history, chunk by chunk, i.e. the
 *                        per-head chunk tensors K^(c)_{l,h} of App. C laid side by side
 *   resident: [n*Bpc]    1 if block b is on the GPU, 0 if it is not (the pointer
 *                        table's 0 entry of App. C / Alg. 1: such blocks are skipped);
 *                        NULL means every block is resident.
 *   Block id b in [0, n*Bpc): chunk c = b div Bpc, offset o = b mod Bpc (Alg. 1, Step 1).
 *
 * Element types: 0 = float64, 1 = float32, 2 = bfloat16 (raw 16-bit patterns).
 * Return value of every entry point: 0 on success, -1 on invalid arguments.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ inputs */

static double widen(const void* base, int64_t i, int et) {
  if (et == 0) return ((const double*)base)[i];
  if (et == 1) return (double)((const float*)base)[i];
  uint32_t bits = ((uint32_t)((const uint16_t*)base)[i]) << 16; /* bf16 is the top half of an fp32 */
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

static int valid_et(int et) { return et == 0 || et == 1 || et == 2; }

/* index of element (chunk c, token t, head h, dim j) in a [n][S][H][d] history tensor */
static int64_t kv_at(int S, int H, int d, int c, int t, int h, int j) {
  return (((int64_t)c * S + t) * H + h) * d + j;
}

/* ------------------------------------------------------------ block geometry */

int oracle_blocks_per_chunk(int S, int B) {
  if (S <= 0 || B <= 0) return -1;
  return (S + B - 1) / B;
}

/* first token (chunk-local) and token count of block offset o within a chunk */
static void block_span(int S, int B, int o, int* first, int* count) {
  int begin = o * B;
  int end = begin + B < S ? begin + B : S;
  *first = begin;
  *count = end - begin;
}

/* ------------------------------------------------------ Adaptive Window Exclusion
 * Sec. 3.2, Eq. 2, with the activation rule of App. B (exclusion starts once
 * enough history lies outside the window).  The window W is the set of blocks of
 * the most recent E chunks.  Exclusion is applied when
 *   (i)  at least T_out whole chunks lie outside the window  (n - E >= T_out), and
 *   (ii) at least K blocks lie outside the window  (|H \ W| = (n - E) * Bpc >= K),
 * condition (ii) being Eq. 2's own guard.  T_out = 0 leaves Eq. 2 alone.
 */
int oracle_awe_active(int n, int E, int T_out, int K, int Bpc) {
  if (n < 0 || E < 0 || T_out < 0 || K < 1 || Bpc < 1) return -1;
  int64_t outside_chunks = (int64_t)n - E;
  if (outside_chunks < 0) outside_chunks = 0;
  int64_t outside_blocks = outside_chunks * Bpc;
  return (outside_chunks >= T_out && outside_blocks >= K) ? 1 : 0;
}

/* Candidate set Omega (Eq. 2): every resident historical block, minus the window
 * blocks when exclusion is active.  omega[b] = 1 for candidates. */
int oracle_candidates(int n, int Bpc, int K, int E, int T_out, const uint8_t* resident, uint8_t* omega) {
  int awe = oracle_awe_active(n, E, T_out, K, Bpc);
  if (awe < 0 || omega == NULL) return -1;
  int64_t nb = (int64_t)n * Bpc;
  for (int64_t b = 0; b < nb; ++b) {
    int c = (int)(b / Bpc);
    int in_window = c >= n - E;
    int is_resident = resident == NULL ? 1 : (resident[b] != 0);
    omega[b] = (uint8_t)(is_resident && !(awe && in_window));
  }
  return awe;
}

/* ------------------------------------------------------------- pooled keys
 * Compression pooling (Sec. 3.1, App. B: a plain mean pool): the pooled key of
 * block b is the mean of the keys of the tokens it holds.  A chunk's last block
 * may hold fewer than B tokens; its mean is over the tokens it holds.
 * kbar: [H][n*Bpc][d]. */
static int pool_heads(int H, int d, int S, int n, int B, int et, const void* K, int h_begin, int h_end,
                      double* kbar) {
  int Bpc = oracle_blocks_per_chunk(S, B);
  if (Bpc < 0 || H < 1 || d < 1 || n < 0 || !valid_et(et) || (n > 0 && K == NULL) || kbar == NULL) return -1;
  int64_t nb = (int64_t)n * Bpc;
#pragma omp parallel for collapse(2) schedule(static)
  for (int h = h_begin; h < h_end; ++h) {
    for (int64_t b = 0; b < nb; ++b) {
      int c = (int)(b / Bpc), o = (int)(b % Bpc), first, count;
      block_span(S, B, o, &first, &count);
      for (int j = 0; j < d; ++j) {
        double sum = 0.0;
        for (int t = first; t < first + count; ++t) sum += widen(K, kv_at(S, H, d, c, t, h, j), et);
        kbar[((int64_t)h * nb + b) * d + j] = sum / count;
      }
    }
  }
  return 0;
}

int oracle_pool_keys(int H, int d, int S, int n, int B, int et, const void* K, double* kbar) {
  return pool_heads(H, d, S, n, B, et, K, 0, H, kbar);
}

/* ----------------------------------------------------------- proxy queries
 * Query-Shared KV Selection (Sec. 3.3, Eq. 3): the chunk's Lq queries are cut into
 * R = ceil(Lq/G_q) groups of adjacent rows, G_r = [r*G_q, min((r+1)*G_q, Lq)).
 * With the score read as the scaled logit against the pooled key, Eq. 3's
 * average of per-query scores over a group equals the score of the group's mean
 * query (linearity), so the proxy query of group r is that mean.
 * qbar: [H][R][d]. */
int oracle_proxy_queries(int H, int d, int Lq, int G_q, int et, const void* Q, double* qbar) {
  if (H < 1 || d < 1 || Lq < 1 || G_q < 1 || !valid_et(et) || Q == NULL || qbar == NULL) return -1;
  int R = (Lq + G_q - 1) / G_q;
#pragma omp parallel for collapse(2) schedule(static)
  for (int h = 0; h < H; ++h) {
    for (int r = 0; r < R; ++r) {
      int q0 = r * G_q, q1 = q0 + G_q < Lq ? q0 + G_q : Lq;
      for (int j = 0; j < d; ++j) {
        double sum = 0.0;
        for (int q = q0; q < q1; ++q) sum += widen(Q, ((int64_t)q * H + h) * d + j, et);
        qbar[(((int64_t)h * R) + r) * d + j] = sum / (q1 - q0);
      }
    }
  }
  return 0;
}

/* Per-query compression scores s_{h,q,b} = scale * (q . kbar_b)  (Eq. 2's input).
 * Used by the tests to check Eq. 3's averaging against the proxy form.
 * s: [H][Lq][n*Bpc]. */
int oracle_query_scores(int H, int d, int S, int n, int B, int Lq, int et_q, const void* Q, int et_k,
                        const void* K, double scale, double* s) {
  int Bpc = oracle_blocks_per_chunk(S, B);
  if (Bpc < 0 || Lq < 1 || !valid_et(et_q) || Q == NULL || s == NULL) return -1;
  int64_t nb = (int64_t)n * Bpc;
  double* kbar = (double*)malloc(sizeof(double) * (size_t)(H * nb * d + 1));
  if (kbar == NULL) return -1;
  if (oracle_pool_keys(H, d, S, n, B, et_k, K, kbar) != 0) { free(kbar); return -1; }
#pragma omp parallel for collapse(2) schedule(static)
  for (int h = 0; h < H; ++h) {
    for (int q = 0; q < Lq; ++q) {
      for (int64_t b = 0; b < nb; ++b) {
        double dot = 0.0;
        for (int j = 0; j < d; ++j) dot += widen(Q, ((int64_t)q * H + h) * d + j, et_q) * kbar[((int64_t)h * nb + b) * d + j];
        s[((int64_t)h * Lq + q) * nb + b] = scale * dot;
      }
    }
  }
  free(kbar);
  return 0;
}

/* ------------------------------------------------------------------ selection
 * Eq. 2 + Eq. 3 for heads [h_begin, h_end):
 *   sbar[h][r][b] = scale * (qbar[h][r] . kbar[h][b])
 *   I[h][r]       = TopK over Omega of sbar[h][r][.]
 * Ranking: higher score first; equal scores rank the lower block id first.
 * Output per (h, r): the min(K, |Omega|) chosen ids in ascending id order,
 * padded with -1 up to K; cnt = number chosen; sel_score = their scores in the
 * same order (padding: -inf).  all_scores (optional) receives sbar for every
 * block, [H][R][n*Bpc], with NaN for blocks outside Omega.
 * Returns the AWE state (0/1) or -1. */
typedef struct {
  double s;
  int32_t b;
} ranked_t;

static int rank_cmp(const void* pa, const void* pb) {
  const ranked_t* a = (const ranked_t*)pa;
  const ranked_t* b = (const ranked_t*)pb;
  if (a->s > b->s) return -1;
  if (a->s < b->s) return 1;
  return (a->b < b->b) ? -1 : (a->b > b->b);
}

static int id_cmp(const void* pa, const void* pb) {
  int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
  return (a > b) - (a < b);
}

int oracle_select(int H, int d, int S, int n, int B, int Lq, int et_q, const void* Q, int et_k, const void* K,
                  const uint8_t* resident, int top_k, int G_q, int E, int T_out, double scale, int h_begin,
                  int h_end, int32_t* idx, int32_t* cnt, double* sel_score, double* all_scores) {
  int Bpc = oracle_blocks_per_chunk(S, B);
  if (Bpc < 0 || H < 1 || d < 1 || n < 0 || Lq < 1 || top_k < 1 || G_q < 1 || E < 0 || T_out < 0) return -1;
  if (h_begin < 0 || h_end > H || h_begin > h_end || idx == NULL || cnt == NULL) return -1;
  if (!valid_et(et_q) || !valid_et(et_k) || Q == NULL || (n > 0 && K == NULL)) return -1;
  int R = (Lq + G_q - 1) / G_q;
  int64_t nb = (int64_t)n * Bpc;

  uint8_t* omega = (uint8_t*)malloc((size_t)nb + 1);
  double* kbar = (double*)malloc(sizeof(double) * (size_t)(H * nb * d + 1));
  double* qbar = (double*)malloc(sizeof(double) * (size_t)(H * R * d));
  if (omega == NULL || kbar == NULL || qbar == NULL) {
    free(omega); free(kbar); free(qbar);
    return -1;
  }
  int awe = oracle_candidates(n, Bpc, top_k, E, T_out, resident, omega);
  int ok = awe >= 0 && pool_heads(H, d, S, n, B, et_k, K, h_begin, h_end, kbar) == 0 &&
           oracle_proxy_queries(H, d, Lq, G_q, et_q, Q, qbar) == 0;
  if (!ok) {
    free(omega); free(kbar); free(qbar);
    return -1;
  }

#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int h = h_begin; h < h_end; ++h) {
    for (int r = 0; r < R; ++r) {
      ranked_t* cand = (ranked_t*)malloc(sizeof(ranked_t) * (size_t)(nb + 1));
      int32_t* chosen = (int32_t*)malloc(sizeof(int32_t) * (size_t)(top_k + 1));
      int64_t m = 0;
      for (int64_t b = 0; b < nb; ++b) {
        double dot = 0.0;
        for (int j = 0; j < d; ++j) dot += qbar[((int64_t)h * R + r) * d + j] * kbar[((int64_t)h * nb + b) * d + j];
        double sb = scale * dot;
        if (all_scores != NULL) all_scores[((int64_t)h * R + r) * nb + b] = omega[b] ? sb : NAN;
        if (omega[b]) {
          cand[m].s = sb;
          cand[m].b = (int32_t)b;
          ++m;
        }
      }
      qsort(cand, (size_t)m, sizeof(ranked_t), rank_cmp);
      int take = m < top_k ? (int)m : top_k;
      for (int t = 0; t < take; ++t) chosen[t] = cand[t].b;
      qsort(chosen, (size_t)take, sizeof(int32_t), id_cmp);
      int64_t base = ((int64_t)h * R + r) * top_k;
      for (int t = 0; t < top_k; ++t) {
        idx[base + t] = t < take ? chosen[t] : -1;
        if (sel_score != NULL) {
          double v = -INFINITY;
          if (t < take) {
            for (int u = 0; u < take; ++u)
              if (cand[u].b == chosen[t]) v = cand[u].s;
          }
          sel_score[base + t] = v;
        }
      }
      cnt[(int64_t)h * R + r] = take;
      free(cand);
      free(chosen);
    }
  }
  free(omega); free(kbar); free(qbar);
  return awe;
}

/* ------------------------------------------------------------------ probability scores
 * The probability-averaged reading of the compression score (Sec. 3.1: selection
 * ranks blocks by the compression branch's attention scores; App. C: that branch
 * attends every pooled token of the history; Eq. 3: a group averages its queries'
 * scores).  For heads [h_begin, h_end), with kc[h] the N = n*Bpc pooled keys:
 *   u[q][b]    = scale * (q . kc[h][b])                 for every pooled token b
 *   p[q][b]    = exp(u[q][b] - LSE_q),  LSE_q = ln sum over all b of exp(u[q][b])
 *   sbar[r][b] = (1/|G_r|) sum over the queries q of group r of p[q][b]
 *   I[h][r]    = TopK over Omega of sbar[r][.]
 * The softmax runs over all N pooled tokens (window and non-resident blocks
 * included); only the top-K is restricted to Omega.  Ranking, output order,
 * padding and all_scores are as in oracle_select.  Returns the AWE state or -1. */
int oracle_select_prob(int H, int d, int n, int Bpc, int Lq, int et_q, const void* Q, const double* kc,
                       const uint8_t* resident, int top_k, int G_q, int E, int T_out, double scale, int h_begin,
                       int h_end, int32_t* idx, int32_t* cnt, double* sel_score, double* all_scores) {
  if (Bpc < 1 || H < 1 || d < 1 || n < 0 || Lq < 1 || top_k < 1 || G_q < 1 || E < 0 || T_out < 0) return -1;
  if (h_begin < 0 || h_end > H || h_begin > h_end || idx == NULL || cnt == NULL) return -1;
  if (!valid_et(et_q) || Q == NULL || (n > 0 && kc == NULL)) return -1;
  int R = (Lq + G_q - 1) / G_q;
  int64_t nb = (int64_t)n * Bpc;
  uint8_t* omega = (uint8_t*)malloc((size_t)nb + 1);
  if (omega == NULL) return -1;
  int awe = oracle_candidates(n, Bpc, top_k, E, T_out, resident, omega);
  if (awe < 0) {
    free(omega);
    return -1;
  }

#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int h = h_begin; h < h_end; ++h) {
    for (int r = 0; r < R; ++r) {
      double* u = (double*)malloc(sizeof(double) * (size_t)(nb + 1));
      double* sbar = (double*)calloc((size_t)(nb + 1), sizeof(double));
      ranked_t* cand = (ranked_t*)malloc(sizeof(ranked_t) * (size_t)(nb + 1));
      int32_t* chosen = (int32_t*)malloc(sizeof(int32_t) * (size_t)(top_k + 1));
      int row0 = r * G_q, row1 = row0 + G_q < Lq ? row0 + G_q : Lq;
      for (int q = row0; q < row1 && nb > 0; ++q) {
        double mx = -INFINITY;
        for (int64_t b = 0; b < nb; ++b) {
          double dot = 0.0;
          for (int j = 0; j < d; ++j) dot += widen(Q, ((int64_t)q * H + h) * d + j, et_q) * kc[((int64_t)h * nb + b) * d + j];
          u[b] = scale * dot;
          mx = u[b] > mx ? u[b] : mx;
        }
        double denom = 0.0;
        for (int64_t b = 0; b < nb; ++b) denom += exp(u[b] - mx);
        double lse_q = mx + log(denom);
        for (int64_t b = 0; b < nb; ++b) sbar[b] += exp(u[b] - lse_q);
      }
      int64_t m = 0;
      for (int64_t b = 0; b < nb; ++b) {
        double sb = sbar[b] / (double)(row1 - row0);
        if (all_scores != NULL) all_scores[((int64_t)h * R + r) * nb + b] = omega[b] ? sb : NAN;
        if (omega[b] != 0) {
          cand[m].s = sb;
          cand[m].b = (int32_t)b;
          ++m;
        }
      }
      qsort(cand, (size_t)m, sizeof(ranked_t), rank_cmp);
      int take = m < top_k ? (int)m : top_k;
      for (int t = 0; t < take; ++t) chosen[t] = cand[t].b;
      qsort(chosen, (size_t)take, sizeof(int32_t), id_cmp);
      int64_t base = ((int64_t)h * R + r) * top_k;
      for (int t = 0; t < top_k; ++t) {
        idx[base + t] = t < take ? chosen[t] : -1;
        if (sel_score != NULL) {
          double v = -INFINITY;
          for (int w = 0; w < take && t < take; ++w)
            if (cand[w].b == chosen[t]) v = cand[w].s;
          sel_score[base + t] = v;
        }
      }
      cnt[(int64_t)h * R + r] = take;
      free(u);
      free(sbar);
      free(cand);
      free(chosen);
    }
  }
  free(omega);
  return awe;
}

/* ------------------------------------------------------------------ attention
 * Softmax attention of one query over an explicit list of key tokens, by the
 * definition: logits u_j = scale * (q . k_j); O = sum_j softmax(u)_j v_j and
 * LSE = ln sum_j exp(u_j), evaluated with the maximum subtracted first.  An empty
 * key set gives O = 0 and LSE = -inf. */
typedef struct {
  int32_t c, t; /* chunk, chunk-local token */
} token_t;

static void attend_one(int H, int d, int S, int et_q, const void* Q, int q, int h, int et_kv, const void* K,
                       const void* V, const token_t* keys, int64_t nkeys, double scale, double* out, double* lse,
                       double* logit_buf) {
  if (nkeys == 0) {
    for (int j = 0; j < d; ++j) out[j] = 0.0;
    *lse = -INFINITY;
    return;
  }
  double mx = -INFINITY;
  for (int64_t i = 0; i < nkeys; ++i) {
    double dot = 0.0;
    for (int j = 0; j < d; ++j)
      dot += widen(Q, ((int64_t)q * H + h) * d + j, et_q) * widen(K, kv_at(S, H, d, keys[i].c, keys[i].t, h, j), et_kv);
    logit_buf[i] = scale * dot;
    if (logit_buf[i] > mx) mx = logit_buf[i];
  }
  double denom = 0.0;
  for (int j = 0; j < d; ++j) out[j] = 0.0;
  for (int64_t i = 0; i < nkeys; ++i) {
    double w = exp(logit_buf[i] - mx);
    denom += w;
    for (int j = 0; j < d; ++j) out[j] += w * widen(V, kv_at(S, H, d, keys[i].c, keys[i].t, h, j), et_kv);
  }
  for (int j = 0; j < d; ++j) out[j] /= denom;
  *lse = mx + log(denom);
}

/* append the tokens of block b (if resident) to keys; returns the new count */
static int64_t push_block(int S, int B, int Bpc, int32_t b, const uint8_t* resident, token_t* keys, int64_t nk) {
  if (resident != NULL && !resident[b]) return nk; /* not resident: skipped (Alg. 1, Step 2) */
  int c = b / Bpc, o = b % Bpc, first, count;
  block_span(S, B, o, &first, &count);
  for (int t = first; t < first + count; ++t) {
    keys[nk].c = c;
    keys[nk].t = t;
    ++nk;
  }
  return nk;
}

/* Selection attention (Alg. 1, Step 2): query q of group r = q div G_q attends to
 * the tokens of the blocks idx[h][r][0:cnt[h][r]], taken in list order (a block
 * listed twice is attended twice, as the loop over the list does); entries < 0
 * are padding.  Computed for m sampled (head, query) pairs (hs[i], qs[i]).
 * out: [m][d], lse: [m]. */
int oracle_sparse_attn(int H, int d, int S, int n, int B, int Lq, int et_q, const void* Q, int et_kv,
                       const void* K, const void* V, const uint8_t* resident, const int32_t* idx,
                       const int32_t* cnt, int top_k, int G_q, double scale, int m, const int32_t* hs,
                       const int32_t* qs, double* out, double* lse) {
  int Bpc = oracle_blocks_per_chunk(S, B);
  if (Bpc < 0 || H < 1 || d < 1 || n < 0 || Lq < 1 || top_k < 1 || G_q < 1 || m < 0) return -1;
  if (!valid_et(et_q) || !valid_et(et_kv) || idx == NULL || cnt == NULL || out == NULL || lse == NULL) return -1;
  int R = (Lq + G_q - 1) / G_q;
  int64_t nb = (int64_t)n * Bpc;
  for (int i = 0; i < m; ++i)
    if (hs[i] < 0 || hs[i] >= H || qs[i] < 0 || qs[i] >= Lq) return -1;
  for (int64_t i = 0; i < (int64_t)H * R; ++i) {
    if (cnt[i] < 0 || cnt[i] > top_k) return -1;
    for (int t = 0; t < cnt[i]; ++t)
      if (idx[i * top_k + t] >= nb) return -1;
  }
  int bad = 0;
#pragma omp parallel for schedule(dynamic)
  for (int i = 0; i < m; ++i) {
    int h = hs[i], q = qs[i], r = q / G_q;
    int64_t row = (int64_t)h * R + r;
    token_t* keys = (token_t*)malloc(sizeof(token_t) * (size_t)((int64_t)top_k * B + 1));
    double* buf = (double*)malloc(sizeof(double) * (size_t)((int64_t)top_k * B + 1));
    if (keys == NULL || buf == NULL) {
      bad = 1;
    } else {
      int64_t nk = 0;
      for (int t = 0; t < cnt[row]; ++t) {
        int32_t b = idx[row * top_k + t];
        if (b < 0) continue;
        nk = push_block(S, B, Bpc, b, resident, keys, nk);
      }
      attend_one(H, d, S, et_q, Q, q, h, et_kv, K, V, keys, nk, scale, out + (int64_t)i * d, lse + i, buf);
    }
    free(keys);
    free(buf);
  }
  return bad ? -1 : 0;
}

/* Dense attention of query q over every resident token of history chunks
 * [c0, c1): c0 = 0, c1 = n is full-history attention; c0 = n - W is the
 * sliding-window branch over the W most recent chunks (App. C). */
int oracle_dense_attn(int H, int d, int S, int n, int B, int Lq, int et_q, const void* Q, int et_kv,
                      const void* K, const void* V, const uint8_t* resident, int c0, int c1, double scale, int m,
                      const int32_t* hs, const int32_t* qs, double* out, double* lse) {
  int Bpc = oracle_blocks_per_chunk(S, B);
  if (Bpc < 0 || H < 1 || d < 1 || n < 0 || Lq < 1 || c0 < 0 || c1 < c0 || c1 > n || m < 0) return -1;
  if (!valid_et(et_q) || !valid_et(et_kv) || out == NULL || lse == NULL) return -1;
  for (int i = 0; i < m; ++i)
    if (hs[i] < 0 || hs[i] >= H || qs[i] < 0 || qs[i] >= Lq) return -1;
  int64_t span = (int64_t)(c1 - c0) * S;
  token_t* keys = (token_t*)malloc(sizeof(token_t) * (size_t)(span + 1));
  if (keys == NULL) return -1;
  int64_t nk = 0;
  for (int32_t b = c0 * Bpc; b < c1 * Bpc; ++b) nk = push_block(S, B, Bpc, b, resident, keys, nk);
  int bad = 0;
#pragma omp parallel for schedule(dynamic)
  for (int i = 0; i < m; ++i) {
    double* buf = (double*)malloc(sizeof(double) * (size_t)(nk + 1));
    if (buf == NULL) {
      bad = 1;
    } else {
      attend_one(H, d, S, et_q, Q, qs[i], hs[i], et_kv, K, V, keys, nk, scale, out + (int64_t)i * d, lse + i, buf);
    }
    free(buf);
  }
  free(keys);
  return bad ? -1 : 0;
}

/* ---------------------------------------------------------------------- union
 * Eq. 4: U_h = union over groups r of I_{h,r}; the cross-head union U = union
 * over h of U_h sets the size of a head-aligned merged buffer (M_merge is
 * proportional to H * |U|), while per-head scattered access touches sum_h |U_h|
 * blocks (Eq. 5).  per_head: [H]; returns |U| through *total. */
int oracle_union(int H, int R, int top_k, int64_t nb, const int32_t* idx, const int32_t* cnt, int32_t* per_head,
                 int32_t* total) {
  if (H < 1 || R < 1 || top_k < 1 || nb < 0 || idx == NULL || cnt == NULL || per_head == NULL || total == NULL)
    return -1;
  uint8_t* any = (uint8_t*)calloc((size_t)nb + 1, 1);
  uint8_t* mine = (uint8_t*)calloc((size_t)nb + 1, 1);
  if (any == NULL || mine == NULL) {
    free(any); free(mine);
    return -1;
  }
  int32_t all = 0;
  for (int h = 0; h < H; ++h) {
    memset(mine, 0, (size_t)nb + 1);
    int32_t count = 0;
    for (int r = 0; r < R; ++r) {
      int64_t row = (int64_t)h * R + r;
      for (int t = 0; t < cnt[row]; ++t) {
        int32_t b = idx[row * top_k + t];
        if (b < 0 || b >= nb) continue;
        if (!mine[b]) { mine[b] = 1; ++count; }
        if (!any[b]) { any[b] = 1; ++all; }
      }
    }
    per_head[h] = count;
  }
  *total = all;
  free(any);
  free(mine);
  return 0;
}

/* Thread count of the OpenMP regions above (timing only; results do not depend on it). */
void oracle_set_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }
int oracle_max_threads(void) { return omp_get_max_threads(); }
