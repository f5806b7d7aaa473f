/*
 * CPU ORACLE for the per-sequence sampling step -- TEST INFRASTRUCTURE ONLY.
 *
 * Only tests/, the smoke check and the benchmark's CPU-baseline leg may load this file's library.
 * The GPU product path never calls it.  It shares no code, header, table or helper with the HIP path.
 *
 * What it computes, per row (paper: sec. 2 "Sampling (T4)" names greedy, top-k and nucleus sampling;
 * sec. 8 "Workload" lists top-p, top-k, min-p, temperature and repetition, presence and frequency
 * penalties; sec. 6 keeps the per-row sampling computation unchanged while rows are split across
 * GPUs, Eq. (opt_sample)).  The paper fixes none of the formulas, so the oracle follows the plain
 * definitions below, in this order, each reading of the paper stated with its step:
 *
 *   O-0  x_v = logit as fp32 (bf16 widened exactly).
 *   O-1  penalties from the row's token history (repetition: the divide-positive / multiply-negative
 *        rule of CTRL, Keskar et al. 2019, the kind of penalty the paper cites from Kulikov et al.;
 *        frequency / presence: the OpenAI API definition the paper cites):
 *          for every v with count c_v > 0:  x = x > 0 ? x / rep : x * rep;
 *                                           x = x - fl(freq * c_v);  x = x - pres      (all fp32)
 *        O-14: with a prompt history as well, the repetition penalty covers every id of the prompt or
 *        the output, and the frequency and presence terms count the output only (c_v = output count).
 *   O-2  temperature T < 1e-5  => greedy: the lowest id among the maxima of x; logprobs use T = 1.
 *   O-3  r = (float)(1 / (double)T);  z_v = fl32(x_v * r), -0 -> +0, -inf stays -inf.
 *   O-4  m = max finite z;  L = log sum exp(z - m)  (double);  logprob_v = z_v - m - L.
 *   O-5  min-p:  tau_m = fl32(m + fl32(log(min(min_p, 1))))  when min_p > 0; keep z >= tau_m.
 *   O-6  top-k:  tau_k = k-th largest z counting duplicates (full sort) when 0 < k < V; keep z >= tau_k.
 *        S2 = finite z kept by both.
 *   O-7  top-p (nucleus, Holtzman et al. 2020) when p < 1: walk S2 by groups of equal z in
 *        descending order accumulating the mass renormalised over S2; the first group reaching p
 *        closes the set; the whole group is kept.  S = S2 if rounding keeps every group below p.
 *   O-8  pi_v = exp(z_v - m) / sum_S exp(z - m)    (double).
 *   O-9  inverse CDF in ascending token id over S: the first v with cumulative pi > u; if rounding
 *        leaves none, the largest v in S with pi_v > 0.
 *   O-10 outputs: id, logprob (O-4, full vocabulary), the n_top largest z (ties -> lower id) with
 *        logprobs, threshold min_{v in S} z_v, |S|, m + log Z_S, dense pi, flags, and two margins
 *        (distance of u to the drawn interval's ends; distance of p to the cumulative masses around
 *        the nucleus cut) that the tests use to exclude rounding-sensitive rows.
 *
 * Build: plain C99, -O2 -ffp-contract=off -fno-fast-math, OpenMP over rows.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define OR_GREEDY 1u
#define OR_EMPTY 2u
#define OR_BAD_INPUT 4u
#define OR_BAD_PARAM 8u

typedef struct {
  const void* logits; /* [B, ld] fp32 or bf16 bit patterns */
  int32_t is_bf16;
  int64_t B, V, ld;
  const float* temperature;
  const int32_t* top_k;
  const float* top_p;
  const float* min_p;
  const float* rep;
  const float* freq;
  const float* pres;
  const int64_t* hist_offsets; /* [B+1] or NULL */
  const int32_t* hist_ids;
  int64_t hist_len; /* entries in hist_ids */
  const float* uniforms; /* [B] or NULL (then no draw: topk/topp only) */
  int32_t n_top;
  /* O-14: a prompt history per row; when given, hist_* holds the row's output tokens only */
  const int64_t* prompt_offsets; /* [B+1] or NULL */
  const int32_t* prompt_ids;
  int64_t prompt_len;
} oracle_in;

typedef struct {
  int32_t* ids;          /* [B] */
  double* logprobs;      /* [B] */
  int32_t* top_ids;      /* [B, n_top] or NULL */
  double* top_logprobs;  /* [B, n_top] or NULL */
  uint32_t* flags;       /* [B] */
  double* cdf_margin;    /* [B] */
  double* topp_margin;   /* [B] */
  double* threshold;     /* [B] min z over S */
  int64_t* kept;         /* [B] |S| */
  double* log_norm;      /* [B] m + log Z_S */
  double* lse;           /* [B] m + L */
  double* probs;         /* [B, V] or NULL */
  float* penalised;      /* [B, V] or NULL: x after O-1 */
} oracle_out;

static float widen_bf16(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

/* Sort key for the full sort: larger z first, then lower id. -inf entries sort last. */
typedef struct {
  float z;
  int32_t id;
} zi_t;

static int cmp_desc(const void* a, const void* b) {
  const zi_t* p = (const zi_t*)a;
  const zi_t* q = (const zi_t*)b;
  if (p->z > q->z) return -1;
  if (p->z < q->z) return 1;
  return (p->id > q->id) - (p->id < q->id);
}

static void sample_row(const oracle_in* in, const oracle_out* out, int64_t i, float* x, float* z,
                       zi_t* ord, int64_t* cnt, unsigned char* inS) {
  const int64_t V = in->V;
  uint32_t flags = 0;

  /* ---- O-0: widen the row ---- */
  if (in->is_bf16) {
    const uint16_t* row = (const uint16_t*)in->logits + i * in->ld;
    for (int64_t v = 0; v < V; ++v) x[v] = widen_bf16(row[v]);
  } else {
    const float* row = (const float*)in->logits + i * in->ld;
    for (int64_t v = 0; v < V; ++v) x[v] = row[v];
  }

  /* ---- per-row parameters; malformed values are flagged and replaced by "off" ---- */
  float T = in->temperature ? in->temperature[i] : 1.0f;
  int32_t k = in->top_k ? in->top_k[i] : 0;
  float p = in->top_p ? in->top_p[i] : 1.0f;
  float mp = in->min_p ? in->min_p[i] : 0.0f;
  float rep = in->rep ? in->rep[i] : 1.0f;
  float freq = in->freq ? in->freq[i] : 0.0f;
  float pres = in->pres ? in->pres[i] : 0.0f;
  if (!isfinite(T)) { flags |= OR_BAD_PARAM; T = 1.0f; }
  if (isnan(p)) { flags |= OR_BAD_PARAM; p = 1.0f; }
  if (isnan(mp)) { flags |= OR_BAD_PARAM; mp = 0.0f; }
  if (!(rep > 0.0f) || isinf(rep)) { flags |= OR_BAD_PARAM; rep = 1.0f; }
  if (!isfinite(freq)) { flags |= OR_BAD_PARAM; freq = 0.0f; }
  if (!isfinite(pres)) { flags |= OR_BAD_PARAM; pres = 0.0f; }

  /* ---- O-1: penalties (O-14: with a prompt history, the repetition penalty covers the tokens of
   * the prompt and of the output, the frequency and presence penalties the output tokens only; inS
   * marks the prompt tokens here and is reused for the kept set below) ---- */
  int have_c = 0, have_p = 0;
  if (in->hist_offsets) {
    int64_t lo = in->hist_offsets[i], hi = in->hist_offsets[i + 1];
    if (lo < 0 || hi < lo || hi > in->hist_len) {
      flags |= OR_BAD_PARAM;
    } else {
      have_c = 1;
      memset(cnt, 0, sizeof(int64_t) * (size_t)V);
      for (int64_t h = lo; h < hi; ++h) {
        int32_t id = in->hist_ids[h];
        if (id < 0 || (int64_t)id >= V) { flags |= OR_BAD_INPUT; continue; }
        cnt[id] += 1;
      }
    }
  }
  if (in->prompt_offsets) {
    int64_t lo = in->prompt_offsets[i], hi = in->prompt_offsets[i + 1];
    if (lo < 0 || hi < lo || hi > in->prompt_len) {
      flags |= OR_BAD_PARAM;
    } else {
      have_p = 1;
      memset(inS, 0, (size_t)V);
      for (int64_t h = lo; h < hi; ++h) {
        int32_t id = in->prompt_ids[h];
        if (id < 0 || (int64_t)id >= V) { flags |= OR_BAD_INPUT; continue; }
        inS[id] = 1;
      }
    }
  }
  if (have_c || have_p) {
    for (int64_t v = 0; v < V; ++v) {
      const int64_t c = have_c ? cnt[v] : 0;
      if (c == 0 && !(have_p && inS[v])) continue;
      float xv = x[v];
      if (xv > 0.0f) xv = xv / rep;
      else xv = xv * rep;
      if (c > 0) {
        float fc = freq * (float)c;
        xv = xv - fc;
        xv = xv - pres;
      }
      x[v] = xv;
    }
  }
  if (out->penalised) memcpy(out->penalised + i * V, x, sizeof(float) * (size_t)V);

  /* ---- O-2 / O-3: greedy test and temperature ---- */
  const int greedy = T < 1e-5f;
  const float r = greedy ? 1.0f : (float)(1.0 / (double)T);
  int any_finite = 0;
  for (int64_t v = 0; v < V; ++v) {
    float xv = x[v];
    float zv;
    if (xv == -INFINITY) zv = -INFINITY;
    else {
      zv = xv * r;
      if (zv == 0.0f) zv = 0.0f; /* -0 -> +0 */
    }
    if (isnan(zv) || zv == INFINITY) flags |= OR_BAD_INPUT;
    if (isfinite(zv)) any_finite = 1;
    z[v] = zv;
  }
  if (greedy) flags |= OR_GREEDY;

  const int32_t nt = in->n_top;
  double* probs = out->probs ? out->probs + i * V : NULL;
  if (probs) for (int64_t v = 0; v < V; ++v) probs[v] = 0.0;
  out->cdf_margin[i] = INFINITY;
  out->topp_margin[i] = INFINITY;

  if (!any_finite) {
    flags |= OR_EMPTY;
    out->ids[i] = -1;
    out->logprobs[i] = -INFINITY;
    out->threshold[i] = -INFINITY;
    out->kept[i] = 0;
    out->log_norm[i] = -INFINITY;
    out->lse[i] = -INFINITY;
    for (int32_t t = 0; t < nt; ++t) {
      out->top_ids[i * nt + t] = -1;
      out->top_logprobs[i * nt + t] = -INFINITY;
    }
    out->flags[i] = flags;
    return;
  }

  /* ---- O-4: max and log-sum-exp over the full vocabulary, in double ---- */
  float m = -INFINITY;
  for (int64_t v = 0; v < V; ++v)
    if (isfinite(z[v]) && z[v] > m) m = z[v];
  double sum = 0.0;
  for (int64_t v = 0; v < V; ++v)
    if (isfinite(z[v])) sum += exp((double)z[v] - (double)m);
  const double L = log(sum);
  out->lse[i] = (double)m + L;

  /* ---- the full sort (descending z, ties by ascending id) ---- */
  for (int64_t v = 0; v < V; ++v) {
    ord[v].z = isfinite(z[v]) ? z[v] : -INFINITY;
    ord[v].id = (int32_t)v;
  }
  qsort(ord, (size_t)V, sizeof(zi_t), cmp_desc);
  int64_t n_fin = 0;
  while (n_fin < V && isfinite(ord[n_fin].z)) ++n_fin;

  /* ---- O-10 (part): top-n by z ---- */
  for (int32_t t = 0; t < nt; ++t) {
    if (t < n_fin) {
      out->top_ids[i * nt + t] = ord[t].id;
      out->top_logprobs[i * nt + t] = (double)ord[t].z - (double)m - L;
    } else {
      out->top_ids[i * nt + t] = -1;
      out->top_logprobs[i * nt + t] = -INFINITY;
    }
  }

  memset(inS, 0, (size_t)V);
  if (greedy) {
    /* lowest id with z == m: the first entry of the sort */
    const int32_t id = ord[0].id;
    inS[id] = 1;
    out->ids[i] = id;
    out->logprobs[i] = (double)z[id] - (double)m - L;
    out->threshold[i] = (double)m;
    out->kept[i] = 1;
    out->log_norm[i] = (double)m; /* m + log(exp(0)) */
    if (probs) probs[id] = 1.0;
    out->flags[i] = flags;
    return;
  }

  /* ---- O-5: min-p ---- */
  float tau_m = -INFINITY;
  if (mp > 0.0f) {
    const float mpc = mp > 1.0f ? 1.0f : mp;
    const float lm = (float)log((double)mpc);
    tau_m = m + lm;
  }
  /* ---- O-6: top-k on the sorted order ---- */
  float tau_k = -INFINITY;
  if (k > 0 && (int64_t)k < V) tau_k = ord[k - 1].z;
  const float tau2 = tau_m > tau_k ? tau_m : tau_k;
  /* S2 = finite and z >= tau2: a prefix of the sorted order */
  int64_t n2 = 0;
  while (n2 < n_fin && ord[n2].z >= tau2) ++n2;

  /* ---- O-7: top-p over S2 by groups of equal z ---- */
  int64_t nS = n2;
  if (p < 1.0f) {
    double Z2 = 0.0;
    for (int64_t t = 0; t < n2; ++t) Z2 += exp((double)ord[t].z - (double)m);
    double c = 0.0, c_prev = 0.0;
    int64_t t = 0;
    int found = 0;
    while (t < n2) {
      int64_t g_end = t;
      double gm = 0.0;
      while (g_end < n2 && ord[g_end].z == ord[t].z) {
        gm += exp((double)ord[g_end].z - (double)m);
        ++g_end;
      }
      c_prev = c;
      c = c + gm / Z2;
      t = g_end;
      if (c >= (double)p) { found = 1; break; }
    }
    if (found) {
      nS = t;
      double a = c - (double)p, b = (double)p - c_prev;
      out->topp_margin[i] = a < b ? a : b;
    } else {
      nS = n2;
      out->topp_margin[i] = (double)p - c; /* cumulative never reached p */
    }
  }

  /* ---- O-8: final distribution over S ---- */
  double ZS = 0.0;
  for (int64_t t = 0; t < nS; ++t) {
    inS[ord[t].id] = 1;
    ZS += exp((double)ord[t].z - (double)m);
  }
  out->threshold[i] = (double)ord[nS - 1].z;
  out->kept[i] = nS;
  out->log_norm[i] = (double)m + log(ZS);
  if (probs)
    for (int64_t t = 0; t < nS; ++t) probs[ord[t].id] = exp((double)ord[t].z - (double)m) / ZS;

  /* ---- O-9: inverse CDF in ascending token id ---- */
  int32_t id = -1;
  if (in->uniforms) {
    const double u = (double)in->uniforms[i];
    double C = 0.0, Cb = 0.0;
    int32_t last_pos = -1;
    double last_b = 0.0, last_a = 0.0;
    for (int64_t v = 0; v < V; ++v) {
      if (!inS[v]) continue;
      const double pv = exp((double)z[v] - (double)m) / ZS;
      Cb = C;
      C = C + pv;
      if (pv > 0.0) { last_pos = (int32_t)v; last_b = Cb; last_a = C; }
      if (C > u) {
        id = (int32_t)v;
        double a = u - Cb, b = C - u;
        out->cdf_margin[i] = a < b ? a : b;
        break;
      }
    }
    if (id < 0) { /* rounding left the cumulative at or below u */
      id = last_pos;
      double a = u - last_b, b = last_a - u;
      out->cdf_margin[i] = a < b ? a : b;
    }
  }
  out->ids[i] = id;
  out->logprobs[i] = id >= 0 ? (double)z[id] - (double)m - L : -INFINITY;
  out->flags[i] = flags;
}

int oracle_sample(const oracle_in* in, const oracle_out* out, int nthreads) {
  if (!in || !out || in->B < 0 || in->V <= 0 || in->ld < in->V) return 1;
  if (in->n_top < 0 || (in->n_top > 0 && (!out->top_ids || !out->top_logprobs))) return 1;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
  int err = 0;
#pragma omp parallel
  {
    const int64_t V = in->V;
    float* x = (float*)malloc(sizeof(float) * (size_t)V);
    float* z = (float*)malloc(sizeof(float) * (size_t)V);
    zi_t* ord = (zi_t*)malloc(sizeof(zi_t) * (size_t)V);
    int64_t* cnt = (int64_t*)malloc(sizeof(int64_t) * (size_t)V);
    unsigned char* inS = (unsigned char*)malloc((size_t)V);
    if (!x || !z || !ord || !cnt || !inS) {
#pragma omp atomic write
      err = 2;
    } else {
#pragma omp for schedule(dynamic, 1)
      for (int64_t i = 0; i < in->B; ++i) sample_row(in, out, i, x, z, ord, cnt, inS);
    }
    free(x); free(z); free(ord); free(cnt); free(inS);
  }
  return err;
}

int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/*
 * O-11 Device random numbers (the paper's deterministic random numbers, sec. 6.2 "Deterministic random
 * number generation": every worker must draw what a single worker would; the paper pre-generates them,
 * the "next" step generates them from a counter instead).  The generator is Philox-4x32 with 10 rounds
 * as published by Salmon, Moraes, Dror and Shaw ("Parallel random numbers: as easy as 1, 2, 3",
 * SC 2011): a round multiplies counter words 0 and 2 by the constants 0xD2511F53 and 0xCD9E8D57 into
 * 64-bit products and recombines the halves with words 1 and 3 and the key; the key advances by the
 * Weyl constants 0x9E3779B9 and 0xBB67AE85 between rounds.
 * The uniform of a row: counter (lo(step), hi(step), lo(seq), hi(seq)), key (lo(seed), hi(seed)),
 * u = (word0 >> 8) * 2^-24, a float in [0, 1).
 */
void oracle_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c[4] = {ctr_in[0], ctr_in[1], ctr_in[2], ctr_in[3]};
  uint32_t k[2] = {key_in[0], key_in[1]};
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k[0] += 0x9E3779B9u;
      k[1] += 0xBB67AE85u;
    }
    const uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c[0];
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c[2];
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    const uint32_t n0 = hi1 ^ c[1] ^ k[0];
    const uint32_t n2 = hi0 ^ c[3] ^ k[1];
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
  }
  out[0] = c[0];
  out[1] = c[1];
  out[2] = c[2];
  out[3] = c[3];
}

void oracle_philox_uniforms(uint64_t seed, uint64_t step, const int64_t* seq_ids, int64_t B, float* out) {
  const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  for (int64_t i = 0; i < B; ++i) {
    const uint64_t seq = seq_ids ? (uint64_t)seq_ids[i] : (uint64_t)i;
    const uint32_t ctr[4] = {(uint32_t)step, (uint32_t)(step >> 32), (uint32_t)seq, (uint32_t)(seq >> 32)};
    uint32_t w[4];
    oracle_philox4x32_10(ctr, key, w);
    out[i] = (float)((double)(w[0] >> 8) * (1.0 / 16777216.0));
  }
}

/*
 * O-12 Early-feedback backfill (sec. 5, "Early-feedback backfill" and "Input processing"): the next
 * iteration's last-token tensor X_T is laid out by the scheduler before sampling ends; the sampler
 * then writes each scheduled sequence's new token into its slot.  Row i's id goes to slot dest[i] when
 * 0 <= dest[i] < n_next; other rows (padding, sequences not scheduled next) are skipped.  Slots named
 * by no row keep their contents.
 */
void oracle_backfill(const int32_t* ids, const int32_t* dest, int64_t B, int32_t* next_tokens, int64_t n_next) {
  for (int64_t i = 0; i < B; ++i) {
    const int64_t d = dest[i];
    if (d >= 0 && d < n_next) next_tokens[d] = ids[i];
  }
}

/*
 * O-13 Rows of the all-to-all receive layout (sec. 6.1, Eq. opt_sample: the exchange written g-hat
 * turns the workers' vocabulary shards into row shards before Sample; sec. 6.2, "Efficient logit
 * exchange").  Worker j receives from every worker w the columns of w's vocabulary shard for j's
 * rows, one block after another, so element v of its row i lies in block v / L at column v % L:
 *     rows[i][v] = buf[(v / L) * S + i * ld + v % L]            (elements of es bytes)
 * L = columns per block, S = elements between block starts, ld = row stride inside a block.  Sampling
 * then runs on these rows unchanged (O-0 to O-10).
 */
void oracle_receive_rows(const void* buf, int32_t es, int64_t B, int64_t V, int64_t ld, int64_t L, int64_t S,
                         void* rows) {
  const unsigned char* src = (const unsigned char*)buf;
  unsigned char* dst = (unsigned char*)rows;
  for (int64_t i = 0; i < B; ++i)
    for (int64_t v = 0; v < V; ++v) {
      const int64_t at = (v / L) * S + i * ld + v % L;
      memcpy(dst + (i * V + v) * es, src + at * es, (size_t)es);
    }
}
