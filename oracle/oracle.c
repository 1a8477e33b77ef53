/*
 * oracle.c -- plain, slow, fp64 CPU oracle for block-sparse causal GQA prefill
 * attention with max-based thresholding and mean correction (FlashPrefill V2).
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may link or call this
 * file; tests, the smoke check and the benchmark's CPU-baseline leg use it to
 * judge the GPU library. It shares no code, header or table with the GPU path.
 *
 * What it computes, per sequence b (length L, n = ceil(L/B) blocks,
 * T_J = [J*B, min((J+1)*B, L))), per KV head h (group size g = Hq/Hkv) and
 * scale = softmax_scale (1/sqrt(d) by default):
 *
 * Prefix KV (chunked prefill, prefix caching): a sequence may hold L_kv >= L
 * keys, of which the L queries are the last ones (query i sits at absolute
 * position P0 + i, P0 = L_kv - L >= 0). Key blocks are then those of the L_kv
 * keys. Query block I covers absolute positions a0 .. a1 (the first and last
 * of its rows), which lie in key blocks Ja = a0/B and Jb = a1/B (Jb = Ja + 1
 * when the block straddles a key-block boundary, which happens when P0 is not
 * a multiple of B). Below, "J <= I" reads J <= Jb, "J == I" (the diagonal)
 * reads Ja <= J <= Jb, "I - J" reads Jb - J, "J < I" (blocks fully visible to
 * every row of the block) reads J < Ja, and "t <= p" uses absolute positions;
 * without a prefix Ja = Jb = I (Sec. 3.3 Eq. page and the varlen execution
 * from (L_q, L_kv); Sec. 4 chunked prefill).
 *
 *  1. Gather k_t, v_t (t < L_kv) through the page table:
 *     slot(b, t) = page_table[b][t / p] * p + t mod p            (Sec. 3.3, Eq. page)
 *  2. Block means kbar_J, vbar_J over T_J in exact fp64          (Sec. 3.2, the
 *     pooled statistics beside Eq. correction).
 *     The scoring key is khat_J = bf16_rne(kbar_J) (precision reading C1).
 *  3. Block score of query block I against key block J <= I: the log of the
 *     block energy summed over every query row of block I (all g heads):
 *         ell[I][J] = log sum_{r in rows(I)} exp(scale * q_r . khat_J)
 *     This is the quantity whose exponential Eq. fused_score accumulates
 *     (running max and base-2 form cancel out), Sec. 3.1 Eq. (1)-(2).
 *  4. Max-based threshold (Sec. 3.1, Eq. select):
 *         mu_I = max_J ell[I][J];   kept iff alpha == 0 or ell >= ln(alpha) + mu_I
 *  5. Forced blocks (Sec. 3.1, Eq. select): sink J < sink_blocks; window
 *     I - J < window_blocks; the diagonal J == I; recent J >= n - recent_blocks;
 *     all restricted to J <= I.
 *     mask byte = kept | forced << 1      (kept includes forced)
 *  6. Attention for each row (p, head) of block I (Sec. 3.2, Eq. correction):
 *         N = sum_{J kept} sum_{t in T_J, t <= p} e^{s_t} v_t
 *             + corr * sum_{J < I, not kept} |T_J| e^{sbar_J} vbar_J
 *         D = same without the values;   O = N / D;   LSE = ln D
 *     with s_t = scale q.k_t and sbar_J = scale q.kbar_J (exact fp64 mean,
 *     precision reading C2). Evaluated with the row maximum subtracted.
 *
 * fp8 inputs (OCP e4m3fn) are decoded exactly and multiplied by their per-head
 * fp32 scale in fp64 before any of the above (Sec. 3.3, Eq. fp8 dequantisation).
 *
 * Query tiles (Sec. 3.3 PackGQA; the selection tile of Eq. csr): by default a
 * query "block" I is the B positions [I*B, (I+1)*B) with all g heads of the
 * KV group (g*B packed rows). With tile_rows = R > 0 it is instead one M-tile
 * of R packed rows, i.e. the Pt = R/g positions [I*Pt, (I+1)*Pt) with all g
 * heads. Its rows lie in key blocks Ja .. Jb exactly as for a query block (one
 * block when P0 is a multiple of B, since Pt divides B; at most two
 * otherwise), and every rule above reads with them. Everything else is
 * unchanged; with R = g*B the two agree.
 *
 * Work is spread over POSIX threads by (b, h, I) unit; every unit is computed
 * independently, so the thread count does not change any result.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int32_t batch, num_q_heads, num_kv_heads, head_dim;
  int32_t block_size, page_size, max_seq_len, max_pages_per_seq;
  double alpha;
  int32_t sink_blocks, window_blocks, recent_blocks, mean_correction;
  double softmax_scale;     /* <= 0: 1/sqrt(head_dim) */
  int32_t dtype;            /* 0: bf16, 1: fp8 e4m3fn */
  int32_t nthreads;         /* <= 0: 1 */
  int32_t max_kv_len;       /* bound of the KV lengths (<= 0: max_seq_len) */
  int32_t tile_rows;        /* packed rows per query tile (<= 0: g * block_size) */
} oracle_params;

/* ---------------- codecs ---------------- */

double oracle_bf16_decode(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

/* Round a double to the nearest bf16 value, ties to even, straight from the
 * double (one rounding). Normal bf16 numbers carry 8 significant bits; below
 * 2^-126 the spacing is fixed at 2^-133. Overflow goes to infinity. */
uint16_t oracle_bf16_encode_rne(double x) {
  if (isnan(x)) return 0x7FC0;
  double ax = fabs(x), r;
  if (ax == 0.0) {
    r = 0.0;
  } else if (ax < ldexp(1.0, -126)) {
    r = ldexp(nearbyint(ldexp(ax, 133)), -133);
  } else {
    int e;
    double f = frexp(ax, &e);               /* ax = f * 2^e, f in [0.5, 1) */
    r = ldexp(nearbyint(ldexp(f, 8)), e - 8);
    double maxv = ldexp(255.0, 127 - 7);    /* (2 - 2^-7) * 2^127 */
    if (r > maxv) r = INFINITY;
  }
  float f32 = (float)r;                     /* exact: r is a bf16 value */
  uint32_t u;
  memcpy(&u, &f32, 4);
  uint16_t out = (uint16_t)(u >> 16);
  if (signbit(x)) out |= 0x8000;
  return out;
}

/* OCP e4m3fn: 1 sign, 4 exponent (bias 7), 3 mantissa bits; no infinities;
 * S.1111.111 is NaN; exponent field 0 encodes subnormals m/8 * 2^-6. */
double oracle_e4m3_decode(uint8_t bits) {
  int s = bits >> 7, e = (bits >> 3) & 15, m = bits & 7;
  double v;
  if (e == 15 && m == 7) return NAN;
  if (e == 0) v = ldexp((double)m / 8.0, -6);
  else v = ldexp(1.0 + (double)m / 8.0, e - 7);
  return s ? -v : v;
}

/* ---------------- context ---------------- */

typedef struct {
  const oracle_params* P;
  const void* q;
  const int32_t* cu;        /* query tokens per sequence */
  const int32_t* cuk;       /* KV tokens per sequence (== cu without a prefix) */
  const void* k;
  const void* v;
  const int32_t* bt;
  const float* qs;
  const float* ks;
  const float* vs;
  int g, d, B, nbmax;       /* nbmax: query tiles (mask rows) */
  int Pt;                   /* positions per query tile (B, or tile_rows / g) */
  int nbk;                  /* key blocks (mask columns, pooled rows) */
  double scale;
  /* pooled statistics [b][Hkv][nbk][d] */
  double* kbar;
  double* vbar;
  double* khat;
  /* work list */
  const int32_t* units;     /* triples (b, h, I) */
  int nunits;
  int next;                 /* atomic cursor */
  pthread_mutex_t lock;
  /* outputs / inputs of the stages */
  uint8_t* mask;            /* [b][Hkv][nbmax][nbk] */
  const uint8_t* mask_in;
  double* ell;              /* [b][Hkv][nbmax][nbk], may be NULL */
  double* mu;               /* [b][Hkv][nbmax], may be NULL */
  double* out;              /* [total][Hq][d] */
  double* lse;              /* [total][Hq], may be NULL */
  int status;
} ctx_t;

static double elem(const ctx_t* c, const void* base, size_t idx, double scale) {
  if (c->P->dtype == 0) return oracle_bf16_decode(((const uint16_t*)base)[idx]);
  return oracle_e4m3_decode(((const uint8_t*)base)[idx]) * scale;
}

/* pool slot of token t of sequence b (Sec. 3.3, Eq. page) */
static size_t slot_of(const ctx_t* c, int b, int t) {
  int p = c->P->page_size;
  if (p == 0) return (size_t)c->cuk[b] + (size_t)t;
  int page = c->bt[(size_t)b * c->P->max_pages_per_seq + t / p];
  return (size_t)page * p + (size_t)(t % p);
}

static void load_q(const ctx_t* c, int b, int pos, int hq, double* out) {
  size_t base = ((size_t)(c->cu[b] + pos) * c->P->num_q_heads + hq) * c->d;
  double sc = c->P->dtype == 1 ? (double)c->qs[hq] : 1.0;
  for (int i = 0; i < c->d; ++i) out[i] = elem(c, c->q, base + i, sc);
}

static void load_kv(const ctx_t* c, const void* base, const float* scales, int b, int h, int t,
                    double* out) {
  size_t off = (slot_of(c, b, t) * c->P->num_kv_heads + h) * c->d;
  double sc = c->P->dtype == 1 ? (double)scales[h] : 1.0;
  for (int i = 0; i < c->d; ++i) out[i] = elem(c, base, off + i, sc);
}

static double dot(const double* a, const double* b, int d) {
  double s = 0.0;
  for (int i = 0; i < d; ++i) s += a[i] * b[i];
  return s;
}

static int seq_len(const ctx_t* c, int b) { return c->cu[b + 1] - c->cu[b]; }
static int kv_len(const ctx_t* c, int b) { return c->cuk[b + 1] - c->cuk[b]; }
/* absolute position of query 0 of sequence b */
static int prefix_of(const ctx_t* c, int b) { return kv_len(c, b) - seq_len(c, b); }

static size_t pool_index(const ctx_t* c, int b, int h, int J) {
  return (((size_t)b * c->P->num_kv_heads + h) * c->nbk + J) * c->d;
}

/* ---------------- step 2: block means ---------------- */

static void pool_bh(ctx_t* c, int b, int h) {
  int L = kv_len(c, b), d = c->d, B = c->B;
  int n = (L + B - 1) / B;
  double* tmp = malloc(sizeof(double) * d);
  for (int J = 0; J < n; ++J) {
    int t0 = J * B, t1 = t0 + B < L ? t0 + B : L;
    double* kb = c->kbar + pool_index(c, b, h, J);
    double* vb = c->vbar + pool_index(c, b, h, J);
    for (int i = 0; i < d; ++i) kb[i] = vb[i] = 0.0;
    for (int t = t0; t < t1; ++t) {
      load_kv(c, c->k, c->ks, b, h, t, tmp);
      for (int i = 0; i < d; ++i) kb[i] += tmp[i];
      load_kv(c, c->v, c->vs, b, h, t, tmp);
      for (int i = 0; i < d; ++i) vb[i] += tmp[i];
    }
    double* kh = c->khat + pool_index(c, b, h, J);
    for (int i = 0; i < d; ++i) {
      kb[i] /= (double)(t1 - t0);
      vb[i] /= (double)(t1 - t0);
      kh[i] = oracle_bf16_decode(oracle_bf16_encode_rne(kb[i]));
    }
  }
  free(tmp);
}

/* ---------------- steps 3-5: score, threshold, force ---------------- */

/* forced blocks of a query block whose rows lie in key blocks Ja .. Jb */
static int forced_block(const ctx_t* c, int n, int Ja, int Jb, int J) {
  const oracle_params* P = c->P;
  if (J > Jb) return 0;
  return J < P->sink_blocks || Jb - J < P->window_blocks || J >= Ja || J >= n - P->recent_blocks;
}

static void estimate_unit(ctx_t* c, int b, int h, int I) {
  const oracle_params* P = c->P;
  int L = seq_len(c, b), d = c->d, B = c->B, g = c->g, Pt = c->Pt;
  int n = (L + Pt - 1) / Pt;                 /* query tiles of the sequence */
  if (I >= n) return;
  int nk = (kv_len(c, b) + B - 1) / B;
  int p0 = I * Pt, p1 = p0 + Pt < L ? p0 + Pt : L;
  int Ja = (prefix_of(c, b) + p0) / B;       /* key blocks of the first and last row */
  int Jb = (prefix_of(c, b) + p1 - 1) / B;
  int rows = (p1 - p0) * g;
  double* qrows = malloc(sizeof(double) * (size_t)rows * d);
  double* x = malloc(sizeof(double) * rows);
  double* ell = malloc(sizeof(double) * (Jb + 1));
  for (int p = p0; p < p1; ++p)
    for (int j = 0; j < g; ++j) load_q(c, b, p, h * g + j, qrows + ((size_t)(p - p0) * g + j) * d);
  double mu = -INFINITY;
  for (int J = 0; J <= Jb; ++J) {
    const double* kh = c->khat + pool_index(c, b, h, J);
    double m = -INFINITY;
    for (int r = 0; r < rows; ++r) {
      x[r] = c->scale * dot(qrows + (size_t)r * d, kh, d);
      if (x[r] > m) m = x[r];
    }
    double s = 0.0;
    for (int r = 0; r < rows; ++r) s += exp(x[r] - m);
    ell[J] = m + log(s);
    if (ell[J] > mu) mu = ell[J];
  }
  size_t row = (((size_t)b * P->num_kv_heads + h) * c->nbmax + I) * c->nbk;
  double la = P->alpha > 0 ? log(P->alpha) : 0.0;
  for (int J = 0; J < c->nbk; ++J) {
    uint8_t byte = 0;
    if (J <= Jb) {
      int thr = P->alpha == 0.0 ? 1 : (ell[J] >= la + mu);
      int f = forced_block(c, nk, Ja, Jb, J);
      byte = (uint8_t)((thr || f) | (f << 1));
      if (c->ell) c->ell[row + J] = ell[J];
    } else if (c->ell) {
      c->ell[row + J] = NAN;
    }
    c->mask[row + J] = byte;
  }
  if (c->mu) c->mu[((size_t)b * P->num_kv_heads + h) * c->nbmax + I] = mu;
  free(qrows);
  free(x);
  free(ell);
}

/* ---------------- step 6: attention with mean correction ---------------- */

static void attend_unit(ctx_t* c, int b, int h, int I) {
  const oracle_params* P = c->P;
  int Lq = seq_len(c, b), d = c->d, B = c->B, g = c->g, Pt = c->Pt;
  int n = (Lq + Pt - 1) / Pt;
  if (I >= n) return;
  int L = kv_len(c, b), P0 = prefix_of(c, b);
  const uint8_t* mrow = c->mask_in + (((size_t)b * P->num_kv_heads + h) * c->nbmax + I) * c->nbk;
  int p0 = I * Pt, p1 = p0 + Pt < Lq ? p0 + Pt : Lq;
  int Ja = (P0 + p0) / B, Jb = (P0 + p1 - 1) / B;   /* key blocks of the first and last row */
  /* keys of the kept blocks, gathered once per unit */
  int nkeys = 0;
  for (int J = 0; J <= Jb; ++J)
    if (mrow[J] & 1) nkeys += (J * B + B < L ? B : L - J * B);
  int* kt = malloc(sizeof(int) * (nkeys + 1));
  double* kk = malloc(sizeof(double) * ((size_t)nkeys + 1) * d);
  double* vv = malloc(sizeof(double) * ((size_t)nkeys + 1) * d);
  int idx = 0;
  for (int J = 0; J <= Jb; ++J) {
    if (!(mrow[J] & 1)) continue;
    int t1 = J * B + B < L ? J * B + B : L;
    for (int t = J * B; t < t1; ++t, ++idx) {
      kt[idx] = t;
      load_kv(c, c->k, c->ks, b, h, t, kk + (size_t)idx * d);
      load_kv(c, c->v, c->vs, b, h, t, vv + (size_t)idx * d);
    }
  }
  /* corrected blocks: J < Ja (fully visible to every row), not kept */
  int ncorr = 0;
  int* cj = malloc(sizeof(int) * (Ja + 1));
  if (P->mean_correction)
    for (int J = 0; J < Ja; ++J)
      if (!(mrow[J] & 1)) cj[ncorr++] = J;
  double* q = malloc(sizeof(double) * d);
  double* lg = malloc(sizeof(double) * ((size_t)nkeys + ncorr + 1));
  double* acc = malloc(sizeof(double) * d);
  for (int p = p0; p < p1; ++p) {
    for (int j = 0; j < g; ++j) {
      int hq = h * g + j;
      load_q(c, b, p, hq, q);
      double m = -INFINITY;
      for (int i = 0; i < nkeys; ++i) {
        lg[i] = kt[i] <= P0 + p ? c->scale * dot(q, kk + (size_t)i * d, d) : -INFINITY;
        if (lg[i] > m) m = lg[i];
      }
      for (int i = 0; i < ncorr; ++i) {
        int J = cj[i];
        int cnt = J * B + B < L ? B : L - J * B;
        lg[nkeys + i] = c->scale * dot(q, c->kbar + pool_index(c, b, h, J), d) + log((double)cnt);
        if (lg[nkeys + i] > m) m = lg[nkeys + i];
      }
      double den = 0.0;
      for (int i = 0; i < d; ++i) acc[i] = 0.0;
      for (int i = 0; i < nkeys + ncorr; ++i) {
        if (lg[i] == -INFINITY) continue;
        double w = exp(lg[i] - m);
        const double* val = i < nkeys ? vv + (size_t)i * d : c->vbar + pool_index(c, b, h, cj[i - nkeys]);
        den += w;
        for (int e = 0; e < d; ++e) acc[e] += w * val[e];
      }
      size_t orow = (size_t)(c->cu[b] + p) * P->num_q_heads + hq;
      for (int e = 0; e < d; ++e) c->out[orow * d + e] = acc[e] / den;
      if (c->lse) c->lse[orow] = m + log(den);
    }
  }
  free(kt); free(kk); free(vv); free(cj); free(q); free(lg); free(acc);
}

/* ---------------- threading ---------------- */

typedef void (*unit_fn)(ctx_t*, int, int, int);
typedef struct { ctx_t* c; unit_fn fn; } job_t;

static void* worker(void* arg) {
  job_t* j = (job_t*)arg;
  ctx_t* c = j->c;
  for (;;) {
    pthread_mutex_lock(&c->lock);
    int u = c->next++;
    pthread_mutex_unlock(&c->lock);
    if (u >= c->nunits) break;
    j->fn(c, c->units[3 * u], c->units[3 * u + 1], c->units[3 * u + 2]);
  }
  return NULL;
}

static void run_units(ctx_t* c, unit_fn fn) {
  int nt = c->P->nthreads > 0 ? c->P->nthreads : 1;
  if (nt > c->nunits) nt = c->nunits > 0 ? c->nunits : 1;
  c->next = 0;
  job_t j = {c, fn};
  pthread_t* th = malloc(sizeof(pthread_t) * nt);
  for (int i = 1; i < nt; ++i) pthread_create(&th[i], NULL, worker, &j);
  worker(&j);
  for (int i = 1; i < nt; ++i) pthread_join(th[i], NULL);
  free(th);
}

static void pool_worker_fn(ctx_t* c, int b, int h, int unused) { (void)unused; pool_bh(c, b, h); }

static int setup(ctx_t* c, const oracle_params* P, const void* q, const int32_t* cu,
                 const int32_t* cuk, const void* k, const void* v, const int32_t* bt,
                 const float* qs, const float* ks, const float* vs) {
  memset(c, 0, sizeof(*c));
  if (P->head_dim <= 0 || P->block_size <= 0 || P->num_kv_heads <= 0 ||
      P->num_q_heads % P->num_kv_heads != 0 || P->batch < 0)
    return 1;
  c->P = P; c->q = q; c->cu = cu; c->cuk = cuk ? cuk : cu; c->k = k; c->v = v; c->bt = bt;
  for (int b = 0; b < P->batch; ++b) {       /* at least as many keys as queries */
    int pre = c->cuk[b + 1] - c->cuk[b] - (c->cu ? c->cu[b + 1] - c->cu[b] : 0);
    if (c->cu && pre < 0) return 1;
  }
  c->qs = qs; c->ks = ks; c->vs = vs;
  c->g = P->num_q_heads / P->num_kv_heads;
  c->d = P->head_dim;
  c->B = P->block_size;
  c->Pt = P->tile_rows > 0 ? P->tile_rows / c->g : P->block_size;
  if (c->Pt <= 0 || c->Pt * c->g != (P->tile_rows > 0 ? P->tile_rows : c->Pt * c->g) ||
      P->block_size % c->Pt != 0)
    return 1;
  c->nbmax = (P->max_seq_len + c->Pt - 1) / c->Pt;
  int maxkv = P->max_kv_len > 0 ? P->max_kv_len : P->max_seq_len;
  c->nbk = (maxkv + P->block_size - 1) / P->block_size;
  c->scale = P->softmax_scale > 0 ? P->softmax_scale : 1.0 / sqrt((double)P->head_dim);
  size_t np = (size_t)P->batch * P->num_kv_heads * (c->nbk > 0 ? c->nbk : 1) * c->d;
  c->kbar = calloc(np, sizeof(double));
  c->vbar = calloc(np, sizeof(double));
  c->khat = calloc(np, sizeof(double));
  pthread_mutex_init(&c->lock, NULL);
  /* pool every (b, h) */
  int npairs = P->batch * P->num_kv_heads;
  int32_t* pairs = malloc(sizeof(int32_t) * 3 * (npairs > 0 ? npairs : 1));
  for (int b = 0; b < P->batch; ++b)
    for (int h = 0; h < P->num_kv_heads; ++h) {
      int i = b * P->num_kv_heads + h;
      pairs[3 * i] = b; pairs[3 * i + 1] = h; pairs[3 * i + 2] = 0;
    }
  c->units = pairs;
  c->nunits = npairs;
  run_units(c, pool_worker_fn);
  free(pairs);
  c->units = NULL;
  c->nunits = 0;
  return 0;
}

static void teardown(ctx_t* c) {
  free(c->kbar); free(c->vbar); free(c->khat);
  pthread_mutex_destroy(&c->lock);
}

/* all (b, h, I) with I < n_b (query tiles), heaviest (largest I) first */
static int32_t* all_units(const ctx_t* c, int* count) {
  const oracle_params* P = c->P;
  int tot = 0;
  for (int b = 0; b < P->batch; ++b) tot += (seq_len(c, b) + c->Pt - 1) / c->Pt * P->num_kv_heads;
  int32_t* u = malloc(sizeof(int32_t) * 3 * (tot > 0 ? tot : 1));
  int i = 0;
  for (int I = c->nbmax - 1; I >= 0; --I)
    for (int b = 0; b < P->batch; ++b) {
      if (I >= (seq_len(c, b) + c->Pt - 1) / c->Pt) continue;
      for (int h = 0; h < P->num_kv_heads; ++h) {
        u[3 * i] = b; u[3 * i + 1] = h; u[3 * i + 2] = I; ++i;
      }
    }
  *count = i;
  return u;
}

/* ---------------- entry points ---------------- */

/* Block means of the KV tokens (cuk: KV lengths): kbar, vbar (fp64) and the
 * bf16 scoring key khat (bit patterns), each [batch][Hkv][nbk][d]; blocks
 * beyond a sequence stay zero. */
int oracle_pool(const oracle_params* P, const void* k, const void* v, const int32_t* bt,
                const int32_t* cuk, const float* ks, const float* vs, double* kbar, double* vbar,
                uint16_t* khat_bits) {
  ctx_t c;
  if (setup(&c, P, NULL, NULL, cuk, k, v, bt, NULL, ks, vs)) return 1;
  size_t np = (size_t)P->batch * P->num_kv_heads * c.nbk * c.d;
  if (kbar) memcpy(kbar, c.kbar, np * sizeof(double));
  if (vbar) memcpy(vbar, c.vbar, np * sizeof(double));
  if (khat_bits)
    for (size_t i = 0; i < np; ++i) khat_bits[i] = oracle_bf16_encode_rne(c.khat[i]);
  teardown(&c);
  return 0;
}

/* Steps 1-5 for the given units (NULL: all). Writes mask rows of those units;
 * ell/mu (optional) receive the block scores and row maxima. */
int oracle_estimate(const oracle_params* P, const void* q, const int32_t* cu, const int32_t* cuk,
                    const void* k, const void* v, const int32_t* bt, const float* qs,
                    const float* ks, const float* vs, const int32_t* units, int nunits,
                    uint8_t* mask, double* ell, double* mu) {
  ctx_t c;
  if (setup(&c, P, q, cu, cuk, k, v, bt, qs, ks, vs)) return 1;
  int32_t* own = NULL;
  if (!units) units = own = all_units(&c, &nunits);
  c.units = units; c.nunits = nunits;
  c.mask = mask; c.ell = ell; c.mu = mu;
  run_units(&c, estimate_unit);
  free(own);
  teardown(&c);
  return 0;
}

/* Step 6 for the given units under an external mask (bit 0 = kept). Writes the
 * fp64 output rows [total][Hq][d] and LSE [total][Hq] of those units. */
int oracle_attend(const oracle_params* P, const void* q, const int32_t* cu, const int32_t* cuk,
                  const void* k, const void* v, const int32_t* bt, const float* qs,
                  const float* ks, const float* vs, const uint8_t* mask_in, const int32_t* units,
                  int nunits, double* out, double* lse) {
  ctx_t c;
  if (setup(&c, P, q, cu, cuk, k, v, bt, qs, ks, vs)) return 1;
  int32_t* own = NULL;
  if (!units) units = own = all_units(&c, &nunits);
  c.units = units; c.nunits = nunits;
  c.mask_in = mask_in; c.out = out; c.lse = lse;
  run_units(&c, attend_unit);
  free(own);
  teardown(&c);
  return 0;
}
