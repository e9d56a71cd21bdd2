/*
 * COVER fp64 CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test-suite, the smoke check and the CPU-baseline leg of the benchmark
 * may load this file.  The product path (the HIP library and its Python binding)
 * never calls it and shares no code, header or table with it.
 *
 * Everything here is plain, slow and written to be checked against the paper by
 * eye: fp64 arithmetic, sequential loops, no blocking, no fusion, and (by the build
 * flag -ffp-contract=off) no fused multiply-add.
 *
 * Paper: "Stop the Flip-Flop: Context-Preserving Verification for Fast Revocable
 * Diffusion Decoding" (arXiv 2602.06161).
 *
 *   cover_oracle_attn            Sec. 5.1 (override memory K',V'; leave-one-out view of a
 *                                seed row), App. B.1: the attention of every query row over
 *                                its own materialised key/value view, full softmax.
 *   cover_oracle_attn_closed     App. B.2-B.4: the paper's post-hoc route -- one attention
 *                                over the overridden memory, then the closed-form diagonal
 *                                correction (delta_i, alpha_i, r_i) for seed rows.
 *   cover_oracle_select          Sec. 5.3: stability-aware score, adaptive budget
 *                                ceil(sqrt(n_t * pi_t)), exclusion, top-k.
 *   cover_oracle_token_stats     Sec. 5.3 (u(j) = -log p_j(y_j)) and Sec. 3 (confidence =
 *                                max probability) from one row of logits.
 *   cover_oracle_attn_stats      Sec. 5.3 (d_in, d_out from the head-averaged last-layer
 *                                attention matrix A).
 *
 * Layouts (all row-major, contiguous):
 *   q, out        [B, Hq,  L, d]        k_*, v_*      [B, Hkv, L, d]
 *   lse           [B, Hq,  L]           seed_idx      [B, max_seeds], n_seed [B]
 * Query head h reads key/value head g = h / (Hq / Hkv).
 *
 * Return codes: 0 ok, 1 invalid sizes, 2 seed contract violated (out of range or
 * duplicate), 3 non-finite / negative selection input, 4 allocation failure.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Threads the OpenMP loops below use (reported with CPU timings), and a way to set them
 * (n > 0; for single-core timings).  Results do not depend on the count. */
int cover_oracle_threads(void) { return omp_get_max_threads(); }
void cover_oracle_set_threads(int n) {
  if (n > 0) omp_set_num_threads(n);
}

#define OR_OK 0
#define OR_ERR_SIZE 1
#define OR_ERR_SEED 2
#define OR_ERR_VALUE 3
#define OR_ERR_ALLOC 4

/* ------------------------------------------------------------------------- */
/* Attention                                                                  */
/* ------------------------------------------------------------------------- */

/* Seed set S_b of one batch row as a membership table (Sec. 3: a set of positions). */
static int seed_table(const int32_t* seed_idx, const int32_t* n_seed, int b, int L,
                      int max_seeds, unsigned char* is_seed) {
  memset(is_seed, 0, (size_t)L);
  int ns = n_seed[b];
  if (ns < 0 || ns > max_seeds) return OR_ERR_SEED;
  for (int t = 0; t < ns; ++t) {
    int j = seed_idx[(size_t)b * max_seeds + t];
    if (j < 0 || j >= L) return OR_ERR_SEED;
    if (is_seed[j]) return OR_ERR_SEED; /* a set has no duplicates */
    is_seed[j] = 1;
  }
  return OR_OK;
}

static double dot(const double* a, const double* b, int d) {
  double s = 0.0;
  for (int k = 0; k < d; ++k) s += a[k] * b[k];
  return s;
}

/* Overridden memory (Sec. 5.1): K'_j = cached K-bar_j for j in S, live K_j otherwise. */
static void build_override(const double* live, const double* cache, const unsigned char* is_seed,
                           int L, int d, double* view) {
  for (int j = 0; j < L; ++j) {
    const double* src = is_seed[j] ? cache : live;
    memcpy(view + (size_t)j * d, src + (size_t)j * d, sizeof(double) * (size_t)d);
  }
}

/* Softmax attention of one query over one key/value view of L rows (Sec. 5.1 / App. B.1):
 *   s_j = scale * <q, K_j>,  w_j = exp(s_j - m) / sum_k exp(s_k - m),
 *   o   = sum_j w_j V_j,     lse = m + log sum_k exp(s_k - m). */
static void attend_row(const double* qi, const double* Kv, const double* Vv, int L, int d,
                       double scale, double* s, double* o, double* lse) {
  double m = -INFINITY;
  for (int j = 0; j < L; ++j) {
    s[j] = scale * dot(qi, Kv + (size_t)j * d, d);
    if (s[j] > m) m = s[j];
  }
  double z = 0.0;
  for (int j = 0; j < L; ++j) z += exp(s[j] - m);
  for (int c = 0; c < d; ++c) o[c] = 0.0;
  for (int j = 0; j < L; ++j) {
    double w = exp(s[j] - m) / z;
    const double* vj = Vv + (size_t)j * d;
    for (int c = 0; c < d; ++c) o[c] += w * vj[c];
  }
  *lse = m + log(z);
}

static int check_sizes(int B, int Hq, int Hkv, int L, int d, int max_seeds) {
  if (B < 0 || Hq <= 0 || Hkv <= 0 || L <= 0 || d <= 0 || max_seeds < 0) return OR_ERR_SIZE;
  if (Hq % Hkv != 0) return OR_ERR_SIZE;
  return OR_OK;
}

/*
 * Materialised leave-one-out attention (Sec. 5.1, App. B.1).
 * rows: flat indices r = (b*Hq + h)*L + i to compute, or NULL for all rows.
 * With rows == NULL, out/lse use the full [B,Hq,L,d] / [B,Hq,L] layout; otherwise out is
 * [n_rows, d] and lse is [n_rows].
 * literal != 0: every row copies its own L x d view (K^(i), V^(i)).
 * literal == 0: rows outside S read the shared override view (which *is* their view);
 *               seed rows still copy theirs.  Same arithmetic in the same order, so
 *               both modes give bitwise-equal results.
 */
int cover_oracle_attn(const double* q, const double* k_live, const double* v_live,
                      const double* k_cache, const double* v_cache,
                      const int32_t* seed_idx, const int32_t* n_seed,
                      int B, int Hq, int Hkv, int L, int d, int max_seeds, double scale,
                      int literal, const int64_t* rows, int64_t n_rows,
                      double* out, double* lse) {
  int rc = check_sizes(B, Hq, Hkv, L, d, max_seeds);
  if (rc) return rc;
  const int group = Hq / Hkv;
  const int64_t total = (int64_t)B * Hq * L;
  const int64_t nr = rows ? n_rows : total;
  for (int64_t r = 0; r < nr; ++r) {
    int64_t f = rows ? rows[r] : r;
    if (f < 0 || f >= total) return OR_ERR_SIZE;
  }
  unsigned char* is_seed = (unsigned char*)malloc((size_t)B * L + 1);
  if (!is_seed) return OR_ERR_ALLOC;
  for (int b = 0; b < B; ++b) {
    rc = seed_table(seed_idx, n_seed, b, L, max_seeds, is_seed + (size_t)b * L);
    if (rc) { free(is_seed); return rc; }
  }
  int failed = 0;
#pragma omp parallel
  {
    double* Kv = (double*)malloc(sizeof(double) * (size_t)L * d);
    double* Vv = (double*)malloc(sizeof(double) * (size_t)L * d);
    double* Ks = (double*)malloc(sizeof(double) * (size_t)L * d);
    double* Vs = (double*)malloc(sizeof(double) * (size_t)L * d);
    double* s = (double*)malloc(sizeof(double) * (size_t)L);
    int64_t shared_bg = -1; /* (b, g) whose override view Ks/Vs currently holds */
    if (!Kv || !Vv || !Ks || !Vs || !s) {
#pragma omp atomic write
      failed = 1;
    } else {
#pragma omp for schedule(dynamic, 4)
      for (int64_t r = 0; r < nr; ++r) {
        int64_t f = rows ? rows[r] : r;
        int i = (int)(f % L);
        int h = (int)((f / L) % Hq);
        int b = (int)(f / ((int64_t)L * Hq));
        int g = h / group;
        const unsigned char* S = is_seed + (size_t)b * L;
        size_t kv_off = ((size_t)b * Hkv + g) * (size_t)L * d;
        const double* qi = q + (((size_t)b * Hq + h) * L + i) * (size_t)d;
        double* oi = out + (size_t)r * d;
        double* li = lse + r;
        const double *Kuse, *Vuse;
        if (literal || S[i]) {
          /* K^(i)_j = K'_j for j != i; K^(i)_i = k_i (live, from the masked input) if i in S. */
          build_override(k_live + kv_off, k_cache + kv_off, S, L, d, Kv);
          build_override(v_live + kv_off, v_cache + kv_off, S, L, d, Vv);
          if (S[i]) {
            memcpy(Kv + (size_t)i * d, k_live + kv_off + (size_t)i * d, sizeof(double) * d);
            memcpy(Vv + (size_t)i * d, v_live + kv_off + (size_t)i * d, sizeof(double) * d);
          }
          Kuse = Kv; Vuse = Vv;
        } else {
          int64_t bg = (int64_t)b * Hkv + g;
          if (bg != shared_bg) {
            build_override(k_live + kv_off, k_cache + kv_off, S, L, d, Ks);
            build_override(v_live + kv_off, v_cache + kv_off, S, L, d, Vs);
            shared_bg = bg;
          }
          Kuse = Ks; Vuse = Vs;
        }
        attend_row(qi, Kuse, Vuse, L, d, scale, s, oi, li);
      }
    }
    free(Kv); free(Vv); free(Ks); free(Vs); free(s);
  }
  free(is_seed);
  return failed ? OR_ERR_ALLOC : OR_OK;
}

/*
 * The paper's own route (App. B.2-B.4): plain attention over the overridden memory
 * K', V' for every row, then for each seed row i
 *   delta_i = <q_i, k_i>/sqrt(d) - <q_i, k'_i>/sqrt(d)   (here with the general scale)
 *   alpha_i = w^ovr_{i,i},  r_i = 1 + alpha_i (exp(delta_i) - 1)
 *   o_i     = (o^ovr_i - alpha_i v'_i + alpha_i exp(delta_i) v_i) / r_i
 * and, since the normaliser becomes Z r_i (Lemma B.1), lse_i = lse^ovr_i + log r_i.
 * Non-seed rows keep o^ovr_i.  Full layout output only.
 */
int cover_oracle_attn_closed(const double* q, const double* k_live, const double* v_live,
                             const double* k_cache, const double* v_cache,
                             const int32_t* seed_idx, const int32_t* n_seed,
                             int B, int Hq, int Hkv, int L, int d, int max_seeds, double scale,
                             double* out, double* lse) {
  int rc = check_sizes(B, Hq, Hkv, L, d, max_seeds);
  if (rc) return rc;
  const int group = Hq / Hkv;
  unsigned char* is_seed = (unsigned char*)malloc((size_t)L + 1);
  double* Kp = (double*)malloc(sizeof(double) * (size_t)L * d);
  double* Vp = (double*)malloc(sizeof(double) * (size_t)L * d);
  int failed = (!is_seed || !Kp || !Vp);
  for (int b = 0; b < B && !failed && !rc; ++b) {
    rc = seed_table(seed_idx, n_seed, b, L, max_seeds, is_seed);
    if (rc) break;
    for (int g = 0; g < Hkv; ++g) {
      size_t kv_off = ((size_t)b * Hkv + g) * (size_t)L * d;
      build_override(k_live + kv_off, k_cache + kv_off, is_seed, L, d, Kp);
      build_override(v_live + kv_off, v_cache + kv_off, is_seed, L, d, Vp);
#pragma omp parallel
      {
        double* s = (double*)malloc(sizeof(double) * (size_t)L);
        if (!s) {
#pragma omp atomic write
          failed = 1;
        } else {
#pragma omp for schedule(dynamic, 8)
          for (int64_t hi = 0; hi < (int64_t)group * L; ++hi) {
            int h = g * group + (int)(hi / L);
            int i = (int)(hi % L);
            size_t row = ((size_t)b * Hq + h) * L + i;
            const double* qi = q + row * d;
            double* oi = out + row * d;
            double lse_ovr;
            attend_row(qi, Kp, Vp, L, d, scale, s, oi, &lse_ovr); /* o^ovr_i, s^ovr_i,: */
            lse[row] = lse_ovr;
            if (!is_seed[i]) continue;
            const double* ki = k_live + kv_off + (size_t)i * d;
            const double* vi = v_live + kv_off + (size_t)i * d;
            const double* vpi = Vp + (size_t)i * d;
            double delta = scale * dot(qi, ki, d) - s[i];
            double alpha = exp(s[i] - lse_ovr); /* w^ovr_{i,i} */
            double ed = exp(delta);
            double r = 1.0 + alpha * (ed - 1.0);
            for (int c = 0; c < d; ++c) oi[c] = (oi[c] - alpha * vpi[c] + alpha * ed * vi[c]) / r;
            lse[row] = lse_ovr + log(r);
          }
        }
        free(s);
      }
      if (failed) break;
    }
  }
  free(is_seed); free(Kp); free(Vp);
  if (rc) return rc;
  return failed ? OR_ERR_ALLOC : OR_OK;
}

/* ------------------------------------------------------------------------- */
/* Seed selection (Sec. 5.3)                                                   */
/* ------------------------------------------------------------------------- */

/* Least r >= 0 with r*r >= c: the integer form of ceil(sqrt(n_t * pi_t)), since
 * n_t * pi_t = n_t (1 - F_t(mean)) is the integer count of scores above the mean. */
static int64_t ceil_isqrt(int64_t c) {
  int64_t r = 0;
  while (r * r < c) ++r;
  return r;
}

/* Larger score first; equal scores: smaller position first. */
static int ranks_before(double sa, int ja, double sb, int jb) {
  if (sa > sb) return 1;
  if (sa < sb) return 0;
  return ja < jb;
}

/*
 * One batch row per call of the inner body; for every row b over region j in [0, Lr):
 *   flags bit 0: j in U_t (unmasked); bit 1: excluded (seed at t-1, or ReMask budget reached).
 *   s_j   = u(j) (1 + d_in(j)) / (1 + d_out(j)),  u(j) = -logp_j          (Sec. 5.3, Score)
 *   mean  = (sum_{j in U} s_j) / n_t, the sum taken as a stride-halving tree over the
 *           region zero-padded to the next power of two
 *   c     = #{j in U : s_j > mean}  (= n_t pi_t, pi_t = 1 - F_t(mean), F_t counts <=)
 *   k     = ceil(sqrt(c)), in integers
 *   E     = U minus the excluded positions; k' = min(k, |E|, max_seeds)
 *   seeds = the k' best of E by (score desc, position asc), emitted ascending by position
 *           plus pos_offset, padded with -1.
 * score (may be NULL): s_j for j in U, 0.0 elsewhere.
 */
int cover_oracle_select(const float* logp, const float* d_in, const float* d_out,
                        const uint8_t* flags, int B, int Lr, int max_seeds, int pos_offset,
                        int32_t* seed_idx, int32_t* n_seed, double* score) {
  if (B < 0 || Lr < 0 || max_seeds < 0) return OR_ERR_SIZE;
  int64_t P = 1;
  while (P < Lr) P *= 2;
  double* a = (double*)malloc(sizeof(double) * (size_t)P);
  double* s = (double*)malloc(sizeof(double) * ((size_t)Lr + 1));
  unsigned char* taken = (unsigned char*)malloc((size_t)Lr + 1);
  if (!a || !s || !taken) { free(a); free(s); free(taken); return OR_ERR_ALLOC; }
  int rc = OR_OK;
  for (int b = 0; b < B && rc == OR_OK; ++b) {
    const size_t base = (size_t)b * Lr;
    int64_t n = 0, n_elig = 0;
    for (int j = 0; j < Lr; ++j) {
      s[j] = 0.0;
      if (!(flags[base + j] & 1u)) continue;
      double lp = (double)logp[base + j], di = (double)d_in[base + j], dv = (double)d_out[base + j];
      if (!isfinite(lp) || !isfinite(di) || !isfinite(dv) || di < 0.0 || dv < 0.0) { rc = OR_ERR_VALUE; break; }
      double u = -lp;
      s[j] = (u * (1.0 + di)) / (1.0 + dv);
      ++n;
      if (!(flags[base + j] & 2u)) ++n_elig;
    }
    if (rc) break;
    if (score) for (int j = 0; j < Lr; ++j) score[base + j] = s[j];
    for (int t = 0; t < max_seeds; ++t) seed_idx[(size_t)b * max_seeds + t] = -1;
    n_seed[b] = 0;
    if (n == 0) continue;
    for (int64_t j = 0; j < P; ++j) a[j] = (j < Lr && (flags[base + j] & 1u)) ? s[j] : 0.0;
    for (int64_t stride = P / 2; stride >= 1; stride /= 2)
      for (int64_t j = 0; j < stride; ++j) a[j] = a[j] + a[j + stride];
    double mean = a[0] / (double)n;
    int64_t c = 0;
    for (int j = 0; j < Lr; ++j)
      if ((flags[base + j] & 1u) && s[j] > mean) ++c;
    int64_t k = ceil_isqrt(c);
    if (k > n_elig) k = n_elig;
    if (k > max_seeds) k = max_seeds;
    /* k rounds of "best remaining eligible position" */
    memset(taken, 0, (size_t)Lr);
    for (int64_t t = 0; t < k; ++t) {
      int best = -1;
      for (int j = 0; j < Lr; ++j) {
        if ((flags[base + j] & 3u) != 1u || taken[j]) continue;
        if (best < 0 || ranks_before(s[j], j, s[best], best)) best = j;
      }
      taken[best] = 1;
    }
    int32_t w = 0;
    for (int j = 0; j < Lr; ++j)
      if (taken[j]) seed_idx[(size_t)b * max_seeds + w++] = j + pos_offset;
    n_seed[b] = w;
  }
  free(a); free(s); free(taken);
  return rc;
}

/* ------------------------------------------------------------------------- */
/* Producers of the selection inputs (Sec. 5.3 signals; Sec. 3 confidence)     */
/* ------------------------------------------------------------------------- */

/*
 * For each of R rows of V logits (row-major [R, V]) and assigned token y[r]:
 *   logp[r] = logit[y] - log sum_v exp(logit[v])          (u = -logp, Sec. 5.3)
 *   conf[r] = max_v p(v) = exp(max_v logit[v] - logsumexp) (Sec. 3 confidence)
 *   amax[r] = the smallest v attaining the maximum logit  (Sec. 3 draft token)
 */
int cover_oracle_token_stats(const double* logits, const int32_t* y, int64_t R, int64_t V,
                             double* logp, double* conf, int32_t* amax) {
  if (R < 0 || V <= 0) return OR_ERR_SIZE;
  for (int64_t r = 0; r < R; ++r)
    if (y[r] < 0 || y[r] >= V) return OR_ERR_SIZE;
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < R; ++r) {
    const double* x = logits + r * V;
    double m = -INFINITY;
    int64_t am = 0;
    for (int64_t v = 0; v < V; ++v)
      if (x[v] > m) { m = x[v]; am = v; }
    double z = 0.0;
    for (int64_t v = 0; v < V; ++v) z += exp(x[v] - m);
    double lz = m + log(z);
    logp[r] = x[y[r]] - lz;
    conf[r] = exp(m - lz);
    amax[r] = (int32_t)am;
  }
  return OR_OK;
}

/*
 * d_in / d_out of Sec. 5.3 from the last layer's attention, averaged over the Hq heads:
 *   A_{q->j} = (1/Hq) sum_h w^(h)_{q,j}, with w the corrected (leave-one-out) weights of
 *   the materialised attention above, each row normalised over all L positions.
 * Over the region [r0, r0 + Lr):
 *   d_in(j)  = sum_{q in region, masked[q]}  A_{q->j}
 *   d_out(j) = sum_{i in region, drafted[i]} A_{j->i}
 * masked, drafted: [B, Lr] bytes (nonzero = member).  Outputs [B, Lr].
 */
int cover_oracle_attn_stats(const double* q, const double* k_live, const double* k_cache,
                            const int32_t* seed_idx, const int32_t* n_seed,
                            int B, int Hq, int Hkv, int L, int d, int max_seeds, double scale,
                            int r0, int Lr, const uint8_t* masked, const uint8_t* drafted,
                            double* d_in, double* d_out) {
  int rc = check_sizes(B, Hq, Hkv, L, d, max_seeds);
  if (rc) return rc;
  if (r0 < 0 || Lr < 0 || r0 + Lr > L) return OR_ERR_SIZE;
  const int group = Hq / Hkv;
  unsigned char* is_seed = (unsigned char*)malloc((size_t)L + 1);
  double* A = (double*)malloc(sizeof(double) * (size_t)Lr * L + 1); /* rows: region queries */
  double* Kp = (double*)malloc(sizeof(double) * (size_t)L * d);
  if (!is_seed || !A || !Kp) { free(is_seed); free(A); free(Kp); return OR_ERR_ALLOC; }
  int failed = 0;
  for (int b = 0; b < B && !rc && !failed; ++b) {
    rc = seed_table(seed_idx, n_seed, b, L, max_seeds, is_seed);
    if (rc) break;
    memset(A, 0, sizeof(double) * (size_t)Lr * L);
    for (int h = 0; h < Hq; ++h) {
      int g = h / group;
      size_t kv_off = ((size_t)b * Hkv + g) * (size_t)L * d;
      build_override(k_live + kv_off, k_cache + kv_off, is_seed, L, d, Kp);
#pragma omp parallel
      {
        double* s = (double*)malloc(sizeof(double) * (size_t)L);
        if (!s) {
#pragma omp atomic write
          failed = 1;
        } else {
#pragma omp for schedule(static)
          for (int rq = 0; rq < Lr; ++rq) {
            int i = r0 + rq;
            const double* qi = q + (((size_t)b * Hq + h) * L + i) * (size_t)d;
            double m = -INFINITY;
            for (int j = 0; j < L; ++j) {
              const double* kj = (j == i && is_seed[i]) ? k_live + kv_off + (size_t)i * d
                                                         : Kp + (size_t)j * d;
              s[j] = scale * dot(qi, kj, d);
              if (s[j] > m) m = s[j];
            }
            double z = 0.0;
            for (int j = 0; j < L; ++j) z += exp(s[j] - m);
            for (int j = 0; j < L; ++j) A[(size_t)rq * L + j] += exp(s[j] - m) / z / (double)Hq;
          }
        }
        free(s);
      }
    }
    for (int j = 0; j < Lr; ++j) {
      double din = 0.0, dout = 0.0;
      for (int rq = 0; rq < Lr; ++rq)
        if (masked[(size_t)b * Lr + rq]) din += A[(size_t)rq * L + (r0 + j)];
      for (int i = 0; i < Lr; ++i)
        if (drafted[(size_t)b * Lr + i]) dout += A[(size_t)j * L + (r0 + i)];
      d_in[(size_t)b * Lr + j] = din;
      d_out[(size_t)b * Lr + j] = dout;
    }
  }
  free(is_seed); free(A); free(Kp);
  if (rc) return rc;
  return failed ? OR_ERR_ALLOC : OR_OK;
}
