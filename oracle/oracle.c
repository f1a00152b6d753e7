/*
 * Plain CPU oracle for the shallow-fusion decode step.
 *
 * TEST INFRASTRUCTURE ONLY: this file is compiled into its own library and is
 * loaded by the tests, by the smoke check and by the benchmark's CPU-baseline
 * leg.  The product library shares no code, header, table or helper with it.
 *
 * What it computes (paper, Sec. III-C, Eq. (1)): for every hypothesis and
 * every vocabulary token y,
 *     score(y) = log p_AM(y|x) + sum_i alpha_i * log p_LM,i(y) + beta * boost(y)
 * with one or more backoff n-gram LMs (each with its own weight alpha_i and
 * its own state; with one LM the weight is written lambda) and a phrase boost,
 * followed by greedy (Sec. III, the decoder emits text greedily) or top-k
 * selection, and the advance of the LM and phrase states.
 *
 * It is written from the plain definitions, not from any fast layout:
 *   - the LM is a set of sorted n-gram tuples searched one tuple at a time;
 *     a conditional is evaluated by the ARPA backoff recursion, token by token;
 *   - the phrase state is the longest suffix of the emitted history that is a
 *     prefix of some phrase, found by comparing suffixes against the sorted
 *     prefix set (brute force, no automaton, no failure links);
 *   - floating point follows a fixed order (one rounding per operation, no
 *     contraction: build with -ffp-contract=off), fp32 for the selection keys,
 *     fp64 for the reference scores.
 *
 * Readings of points the paper leaves open (all documented with the build):
 *   LM tables are natural-log; blank never receives LM or boost terms;
 *   mode A (greedy default): the acoustic argmax decides blank vs. emit and the
 *   fused score re-ranks the non-blank tokens; mode B: blank competes with key
 *   x_blank; ties go to the lowest token id; the boost is a potential
 *   difference over phrase prefixes (see score_row below); the LM terms are
 *   added in the order the models are given, before the boost term.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#define OR_MAXN 16
#define OR_MAXLM 4 /* LMs per call */
#define OR_OK 0
#define OR_EARG (-1)
#define OR_ENOMEM (-2)
#define OR_EFORMAT (-4)
#define OR_EPHRASES (-5)

static __thread char g_err[256];
const char *or_last_error(void) { return g_err; }
static int fail(int code, const char *msg) {
  snprintf(g_err, sizeof g_err, "%s", msg);
  return code;
}

/* ------------------------------------------------------------------------ */
/* tuples                                                                    */
/* ------------------------------------------------------------------------ */
static int cmp_tuple(const int32_t *a, const int32_t *b, int k) {
  for (int i = 0; i < k; ++i) {
    if (a[i] < b[i]) return -1;
    if (a[i] > b[i]) return 1;
  }
  return 0;
}

/* rows of k tokens, sorted lexicographically: index of t or -1 */
static int64_t find_row(const int32_t *rows, int64_t n, int k, const int32_t *t) {
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    int64_t mid = lo + (hi - lo) / 2;
    int c = cmp_tuple(rows + mid * (int64_t)k, t, k);
    if (c == 0) return mid;
    if (c < 0) lo = mid + 1;
    else hi = mid;
  }
  return -1;
}

/* qsort helpers: sort a permutation of row indices (single-threaded use only) */
static const int32_t *g_sort_rows;
static int g_sort_k;
static int cmp_perm(const void *pa, const void *pb) {
  int64_t a = *(const int64_t *)pa, b = *(const int64_t *)pb;
  int c = cmp_tuple(g_sort_rows + a * g_sort_k, g_sort_rows + b * g_sort_k, g_sort_k);
  if (c) return c;
  return (a > b) - (a < b);
}

/* ------------------------------------------------------------------------ */
/* n-gram LM                                                                  */
/* ------------------------------------------------------------------------ */
typedef struct OrLM {
  int N, V, blank;
  int64_t n[OR_MAXN + 1];
  int32_t *tok[OR_MAXN + 1]; /* order k: n[k] rows of k tokens, sorted */
  float *lp[OR_MAXN + 1];
  float *bo[OR_MAXN + 1];    /* 0 where the input gave none */
  int64_t off[OR_MAXN + 2];  /* state ids: unigram context w -> w; order k -> off[k] + row */
  int64_t n_states;
} OrLM;

void or_lm_free(OrLM *lm) {
  if (!lm) return;
  for (int k = 1; k <= OR_MAXN; ++k) {
    free(lm->tok[k]);
    free(lm->lp[k]);
    free(lm->bo[k]);
  }
  free(lm);
}

OrLM *or_lm_new(int N, int V, int blank, const int64_t *count, const int32_t *const *tokens,
                const float *const *logp, const float *const *backoff) {
  g_err[0] = 0;
  if (N < 2 || N > OR_MAXN || V < 2 || blank < 0 || blank >= V || !count || !tokens || !logp) {
    fail(OR_EARG, "bad LM arguments");
    return NULL;
  }
  OrLM *lm = (OrLM *)calloc(1, sizeof(OrLM));
  if (!lm) return NULL;
  lm->N = N;
  lm->V = V;
  lm->blank = blank;
  for (int k = 1; k <= N; ++k) {
    int64_t n = count[k - 1];
    if (n < 0 || (n > 0 && (!tokens[k - 1] || !logp[k - 1]))) {
      fail(OR_EARG, "missing order table");
      or_lm_free(lm);
      return NULL;
    }
    lm->n[k] = n;
    lm->tok[k] = (int32_t *)malloc((size_t)(n * k + 1) * sizeof(int32_t));
    lm->lp[k] = (float *)malloc((size_t)(n + 1) * sizeof(float));
    lm->bo[k] = (float *)calloc((size_t)(n + 1), sizeof(float));
    int64_t *perm = (int64_t *)malloc((size_t)(n + 1) * sizeof(int64_t));
    if (!lm->tok[k] || !lm->lp[k] || !lm->bo[k] || !perm) {
      free(perm);
      fail(OR_ENOMEM, "out of host memory");
      or_lm_free(lm);
      return NULL;
    }
    const int32_t *src = tokens[k - 1];
    int sorted = 1;
    for (int64_t i = 0; i < n; ++i) {
      perm[i] = i;
      for (int j = 0; j < k; ++j) {
        int32_t t = src[i * k + j];
        if (t < 0 || t >= V + 2 || t == blank) {
          free(perm);
          fail(OR_EFORMAT, "n-gram token out of range or blank");
          or_lm_free(lm);
          return NULL;
        }
      }
      if (i > 0 && cmp_tuple(src + (i - 1) * k, src + i * k, k) >= 0) sorted = 0;
    }
    if (!sorted) {
      g_sort_rows = src;
      g_sort_k = k;
      qsort(perm, (size_t)n, sizeof(int64_t), cmp_perm);
    }
    for (int64_t i = 0; i < n; ++i) {
      int64_t s = perm[i];
      memcpy(lm->tok[k] + i * k, src + s * k, (size_t)k * sizeof(int32_t));
      float p = logp[k - 1][s];
      float b = (backoff && k < N && backoff[k - 1]) ? backoff[k - 1][s] : 0.0f;
      if (!isfinite(p) || !isfinite(b)) {
        free(perm);
        fail(OR_EFORMAT, "non-finite log-probability or backoff");
        or_lm_free(lm);
        return NULL;
      }
      lm->lp[k][i] = p;
      lm->bo[k][i] = b;
      if (i > 0 && cmp_tuple(lm->tok[k] + (i - 1) * k, lm->tok[k] + i * k, k) == 0) {
        free(perm);
        fail(OR_EFORMAT, "duplicate n-gram");
        or_lm_free(lm);
        return NULL;
      }
    }
    free(perm);
  }
  /* every non-blank id and <s> must have a unigram */
  for (int32_t w = 0; w < V + 1; ++w) {
    if (w == blank) continue;
    if (find_row(lm->tok[1], lm->n[1], 1, &w) < 0) {
      fail(OR_EFORMAT, "missing unigram");
      or_lm_free(lm);
      return NULL;
    }
  }
  lm->off[1] = 0;
  lm->off[2] = V + 2;
  for (int k = 2; k <= N; ++k) lm->off[k + 1] = lm->off[k] + lm->n[k];
  lm->n_states = lm->off[N]; /* orders 1..N-1 are contexts; order N never is */
  return lm;
}

int64_t or_lm_n_states(const OrLM *lm) { return lm->n_states; }

/* is the tuple t[0..k) an n-gram of the model? */
static int64_t lm_find(const OrLM *lm, const int32_t *t, int k) {
  if (k < 1 || k > lm->N) return -1;
  return find_row(lm->tok[k], lm->n[k], k, t);
}

/* state id -> tuple (oldest first); returns length or -1 for an invalid id */
int or_lm_state_tuple(const OrLM *lm, int64_t id, int32_t *out) {
  if (id < 0 || id >= lm->n_states) return -1;
  if (id < lm->V + 2) {
    int32_t w = (int32_t)id;
    if (lm_find(lm, &w, 1) < 0) return -1;
    out[0] = w;
    return 1;
  }
  for (int k = 2; k <= lm->N - 1; ++k) {
    if (id >= lm->off[k] && id < lm->off[k] + lm->n[k]) {
      memcpy(out, lm->tok[k] + (id - lm->off[k]) * k, (size_t)k * sizeof(int32_t));
      return k;
    }
  }
  return -1;
}

/* the state of history h[0..len): its longest suffix of at most N-1 tokens
   that is an n-gram of the model (the last token alone always is) */
int64_t or_lm_state_of_history(const OrLM *lm, const int32_t *h, int len) {
  int top = len < lm->N - 1 ? len : lm->N - 1;
  for (int L = top; L >= 1; --L) {
    int64_t r = lm_find(lm, h + len - L, L);
    if (r >= 0) return L == 1 ? (int64_t)h[len - 1] : lm->off[L] + r;
  }
  return -1;
}

/* backoff of context c (0 when c is not an n-gram of the model) */
static float lm_bo32(const OrLM *lm, const int32_t *c, int len) {
  int64_t r = lm_find(lm, c, len);
  return r >= 0 ? lm->bo[len][r] : 0.0f;
}

/* ARPA backoff, right-recursive, fp32 with one rounding per addition:
   lm(y|c) = p*(c y) if (c y) is an n-gram, else lm(y|c[1:]) + bo(c);
   lm(y|empty) = p*(y).  c holds at most N-1 tokens. */
float or_lm_logp32(const OrLM *lm, const int32_t *c, int len, int32_t y) {
  int32_t t[OR_MAXN + 1];
  memcpy(t, c, (size_t)len * sizeof(int32_t));
  t[len] = y;
  int64_t r = lm_find(lm, t, len + 1);
  if (r >= 0) return lm->lp[len + 1][r];
  if (len == 0) return NAN; /* no unigram: never for a validated model */
  float lower = or_lm_logp32(lm, c + 1, len - 1, y);
  float b = lm_bo32(lm, c, len);
  return lower + b;
}

/* the same recursion carried in fp64 over the stored fp32 values */
double or_lm_logp64(const OrLM *lm, const int32_t *c, int len, int32_t y) {
  int32_t t[OR_MAXN + 1];
  memcpy(t, c, (size_t)len * sizeof(int32_t));
  t[len] = y;
  int64_t r = lm_find(lm, t, len + 1);
  if (r >= 0) return (double)lm->lp[len + 1][r];
  if (len == 0) return NAN;
  return or_lm_logp64(lm, c + 1, len - 1, y) + (double)lm_bo32(lm, c, len);
}

/* the whole conditional row over every LM token id 0..V+1 (fp64 recursion);
   blank and <s> are never predicted and get NaN */
void or_lm_row64(const OrLM *lm, const int32_t *c, int len, double *out) {
  for (int32_t y = 0; y < lm->V + 2; ++y)
    out[y] = (y == lm->blank || y == lm->V) ? NAN : or_lm_logp64(lm, c, len, y);
}

/* ------------------------------------------------------------------------ */
/* phrase boost                                                               */
/* ------------------------------------------------------------------------ */
typedef struct OrTrie {
  int V, blank, maxlen;
  float ts;
  int64_t n_phr;      /* distinct phrases, sorted by (length, tokens) */
  int32_t *phr;       /* [n_phr * maxlen], padded with -1 */
  int32_t *phr_len;
  float *comp;        /* completion bonus c_p */
  int64_t n_nodes;    /* distinct prefixes incl. the empty one, sorted by (length, tokens) */
  int32_t *node;      /* [n_nodes * maxlen] */
  int32_t *node_len;
  float *phi, *E;     /* fp32 potential and entry value per node */
  double *phi64, *E64;
} OrTrie;

void or_trie_free(OrTrie *t) {
  if (!t) return;
  free(t->phr);
  free(t->phr_len);
  free(t->comp);
  free(t->node);
  free(t->node_len);
  free(t->phi);
  free(t->E);
  free(t->phi64);
  free(t->E64);
  free(t);
}

/* (length, lexicographic) order on padded rows */
static int cmp_len_lex(const int32_t *a, int la, const int32_t *b, int lb) {
  if (la != lb) return la < lb ? -1 : 1;
  return cmp_tuple(a, b, la);
}
static const int32_t *g_ll_rows;
static const int32_t *g_ll_len;
static int g_ll_w;
static int cmp_perm_ll(const void *pa, const void *pb) {
  int64_t a = *(const int64_t *)pa, b = *(const int64_t *)pb;
  int c = cmp_len_lex(g_ll_rows + a * g_ll_w, g_ll_len[a], g_ll_rows + b * g_ll_w, g_ll_len[b]);
  if (c) return c;
  return (a > b) - (a < b); /* stable: the earlier input row first */
}

static int64_t find_ll(const int32_t *rows, const int32_t *lens, int64_t n, int w, const int32_t *t,
                       int len) {
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    int64_t mid = lo + (hi - lo) / 2;
    int c = cmp_len_lex(rows + mid * w, lens[mid], t, len);
    if (c == 0) return mid;
    if (c < 0) lo = mid + 1;
    else hi = mid;
  }
  return -1;
}

int64_t or_trie_phrase_index(const OrTrie *t, const int32_t *p, int len) {
  if (len < 1 || len > t->maxlen) return -1;
  return find_ll(t->phr, t->phr_len, t->n_phr, t->maxlen, p, len);
}
/* node id of prefix p (the empty prefix is node 0), or -1 */
int64_t or_trie_node_of(const OrTrie *t, const int32_t *p, int len) {
  if (len < 0 || len > t->maxlen) return -1;
  return find_ll(t->node, t->node_len, t->n_nodes, t->maxlen, p, len);
}
int or_trie_node_tuple(const OrTrie *t, int64_t id, int32_t *out) {
  if (id < 0 || id >= t->n_nodes) return -1;
  int len = t->node_len[id];
  memcpy(out, t->node + id * t->maxlen, (size_t)len * sizeof(int32_t));
  return len;
}
int64_t or_trie_n_nodes(const OrTrie *t) { return t->n_nodes; }
int or_trie_max_len(const OrTrie *t) { return t->maxlen; }
float or_trie_phi(const OrTrie *t, int64_t id) { return t->phi[id]; }
float or_trie_entry(const OrTrie *t, int64_t id) { return t->E[id]; }

OrTrie *or_trie_new(int V, int blank, int64_t n, const int32_t *tokens, const int64_t *offsets,
                    const float *completion, float ts) {
  g_err[0] = 0;
  if (V < 2 || blank < 0 || blank >= V || n < 0 || (n > 0 && (!tokens || !offsets))) {
    fail(OR_EARG, "bad phrase arguments");
    return NULL;
  }
  int maxlen = 0;
  for (int64_t i = 0; i < n; ++i) {
    int64_t L = offsets[i + 1] - offsets[i];
    if (L < 1 || L > 4096) {
      fail(OR_EPHRASES, "empty or overlong phrase");
      return NULL;
    }
    for (int64_t j = offsets[i]; j < offsets[i + 1]; ++j)
      if (tokens[j] < 0 || tokens[j] >= V || tokens[j] == blank) {
        fail(OR_EPHRASES, "phrase token out of range or blank");
        return NULL;
      }
    if (L > maxlen) maxlen = (int)L;
  }
  if (maxlen == 0) maxlen = 1;
  OrTrie *t = (OrTrie *)calloc(1, sizeof(OrTrie));
  t->V = V;
  t->blank = blank;
  t->maxlen = maxlen;
  t->ts = ts;
  /* phrases sorted by (length, tokens); duplicates keep the earliest input */
  int32_t *rows = (int32_t *)malloc((size_t)(n + 1) * maxlen * sizeof(int32_t));
  int32_t *lens = (int32_t *)malloc((size_t)(n + 1) * sizeof(int32_t));
  int64_t *perm = (int64_t *)malloc((size_t)(n + 1) * sizeof(int64_t));
  for (int64_t i = 0; i < n; ++i) {
    int L = (int)(offsets[i + 1] - offsets[i]);
    lens[i] = L;
    for (int j = 0; j < maxlen; ++j) rows[i * maxlen + j] = j < L ? tokens[offsets[i] + j] : -1;
    perm[i] = i;
  }
  g_ll_rows = rows;
  g_ll_len = lens;
  g_ll_w = maxlen;
  qsort(perm, (size_t)n, sizeof(int64_t), cmp_perm_ll);
  t->phr = (int32_t *)malloc((size_t)(n + 1) * maxlen * sizeof(int32_t));
  t->phr_len = (int32_t *)malloc((size_t)(n + 1) * sizeof(int32_t));
  t->comp = (float *)malloc((size_t)(n + 1) * sizeof(float));
  int64_t m = 0;
  for (int64_t i = 0; i < n; ++i) {
    int64_t s = perm[i];
    if (m > 0 && cmp_len_lex(t->phr + (m - 1) * maxlen, t->phr_len[m - 1], rows + s * maxlen,
                             lens[s]) == 0)
      continue; /* same phrase again: the first one's bonus stays */
    memcpy(t->phr + m * maxlen, rows + s * maxlen, (size_t)maxlen * sizeof(int32_t));
    t->phr_len[m] = lens[s];
    t->comp[m] = completion ? completion[s] : ts * (float)lens[s];
    ++m;
  }
  t->n_phr = m;
  /* all prefixes (including the empty one), sorted by (length, tokens), distinct */
  int64_t total = 1;
  for (int64_t i = 0; i < m; ++i) total += t->phr_len[i];
  int32_t *prow = (int32_t *)malloc((size_t)total * maxlen * sizeof(int32_t));
  int32_t *plen = (int32_t *)malloc((size_t)total * sizeof(int32_t));
  int64_t *pperm = (int64_t *)malloc((size_t)total * sizeof(int64_t));
  int64_t c = 0;
  for (int j = 0; j < maxlen; ++j) prow[j] = -1;
  plen[0] = 0;
  c = 1;
  for (int64_t i = 0; i < m; ++i)
    for (int L = 1; L <= t->phr_len[i]; ++L) {
      for (int j = 0; j < maxlen; ++j) prow[c * maxlen + j] = j < L ? t->phr[i * maxlen + j] : -1;
      plen[c] = L;
      ++c;
    }
  for (int64_t i = 0; i < total; ++i) pperm[i] = i;
  g_ll_rows = prow;
  g_ll_len = plen;
  g_ll_w = maxlen;
  qsort(pperm, (size_t)total, sizeof(int64_t), cmp_perm_ll);
  t->node = (int32_t *)malloc((size_t)total * maxlen * sizeof(int32_t));
  t->node_len = (int32_t *)malloc((size_t)total * sizeof(int32_t));
  int64_t nn = 0;
  for (int64_t i = 0; i < total; ++i) {
    int64_t s = pperm[i];
    if (nn > 0 && cmp_len_lex(t->node + (nn - 1) * maxlen, t->node_len[nn - 1], prow + s * maxlen,
                              plen[s]) == 0)
      continue;
    memcpy(t->node + nn * maxlen, prow + s * maxlen, (size_t)maxlen * sizeof(int32_t));
    t->node_len[nn] = plen[s];
    ++nn;
  }
  t->n_nodes = nn;
  free(rows);
  free(lens);
  free(perm);
  free(prow);
  free(plen);
  free(pperm);
  /* potential: 0 at a complete phrase, depth * token_score elsewhere;
     out: completion bonuses of every phrase that is a suffix of the node,
     accumulated from the shortest suffix up; entry value E = phi + out */
  t->phi = (float *)malloc((size_t)nn * sizeof(float));
  t->E = (float *)malloc((size_t)nn * sizeof(float));
  t->phi64 = (double *)malloc((size_t)nn * sizeof(double));
  t->E64 = (double *)malloc((size_t)nn * sizeof(double));
  for (int64_t q = 0; q < nn; ++q) {
    const int32_t *p = t->node + q * maxlen;
    int len = t->node_len[q];
    int complete = or_trie_phrase_index(t, p, len) >= 0;
    float phi = complete ? 0.0f : (float)len * ts;
    double phi64 = complete ? 0.0 : (double)len * (double)ts;
    float out = 0.0f;
    double out64 = 0.0;
    for (int L = 1; L <= len; ++L) {
      int64_t pi = or_trie_phrase_index(t, p + len - L, L);
      if (pi >= 0) {
        out = t->comp[pi] + out;
        out64 = (double)t->comp[pi] + out64;
      }
    }
    t->phi[q] = phi;
    t->phi64[q] = phi64;
    t->E[q] = phi + out;
    t->E64[q] = phi64 + out64;
  }
  return t;
}

/* phrase state after history h[0..len): the longest suffix of h that is a
   prefix of some phrase (node 0 when none), by direct comparison */
int64_t or_trie_state_of_history(const OrTrie *t, const int32_t *h, int len) {
  int top = len < t->maxlen ? len : t->maxlen;
  for (int L = top; L >= 1; --L) {
    int64_t q = or_trie_node_of(t, h + len - L, L);
    if (q >= 0) return q;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* one hypothesis, one frame                                                  */
/* ------------------------------------------------------------------------ */
typedef struct {
  const OrLM *lm[OR_MAXLM];
  float lam[OR_MAXLM]; /* alpha_i of each LM */
  int n_lm;
  const OrTrie *tr;
  int V, blank, k, mode;
  float beta;
  int recombine; /* beam: merge candidates that reach the same history */
} Ctx;

/* Histories: the context of LM i is the last <= N_i-1 tokens of its history
   (<s> or the tuple of its incoming state, then the emitted tokens); the
   phrase history is the emitted tokens (or, step-wise, the tuple of the
   incoming state).  Fills key32[V], f64[V] (fused reference score), next_q[V]
   (phrase state after y); returns lse in fp64. */
static double score_row(const Ctx *c, const float *x, int32_t *const *lmh, const int *lmlen,
                        const int32_t *ph, int plen, float *key32, double *f64, int64_t *next_q) {
  int V = c->V;
  double m = -INFINITY;
  for (int y = 0; y < V; ++y) m = (double)x[y] > m ? (double)x[y] : m;
  double s = 0.0;
  for (int y = 0; y < V; ++y) s += exp((double)x[y] - m);
  double lse = m + log(s);
  const int32_t *ctx[OR_MAXLM];
  int clen[OR_MAXLM];
  for (int i = 0; i < c->n_lm; ++i) {
    int N1 = c->lm[i]->N - 1;
    ctx[i] = lmlen[i] > N1 ? lmh[i] + (lmlen[i] - N1) : lmh[i];
    clen[i] = lmlen[i] > N1 ? N1 : lmlen[i];
  }
  /* current phrase state and its potential */
  int64_t q = c->tr ? or_trie_state_of_history(c->tr, ph, plen) : 0;
  float phi_q = c->tr ? c->tr->phi[q] : 0.0f;
  double phi_q64 = c->tr ? c->tr->phi64[q] : 0.0;
  int32_t *buf = (int32_t *)malloc((size_t)(plen + 1) * sizeof(int32_t));
  memcpy(buf, ph, (size_t)plen * sizeof(int32_t));
  for (int y = 0; y < V; ++y) {
    if (y == c->blank) {
      key32[y] = x[y];
      f64[y] = (double)x[y] - lse;
      next_q[y] = q;
      continue;
    }
    /* the LM terms in model order: u = fl(... fl(x + fl(a_1 l_1)) ... + fl(a_n l_n)) */
    float u = x[y];
    double acc64 = (double)x[y] - lse;
    for (int i = 0; i < c->n_lm; ++i) {
      float l32 = or_lm_logp32(c->lm[i], ctx[i], clen[i], y);
      double l64 = or_lm_logp64(c->lm[i], ctx[i], clen[i], y);
      float a = c->lam[i] * l32;
      u = u + a;
      acc64 = acc64 + (double)c->lam[i] * l64;
    }
    float b32 = 0.0f;
    double b64 = 0.0;
    int64_t nq = 0;
    if (c->tr) {
      buf[plen] = y;
      nq = or_trie_state_of_history(c->tr, buf, plen + 1);
      b32 = c->tr->E[nq] - phi_q;
      b64 = c->tr->E64[nq] - phi_q64;
    }
    float v = c->beta * b32;
    key32[y] = u + v;
    f64[y] = acc64 + (double)c->beta * b64;
    next_q[y] = nq;
  }
  free(buf);
  return lse;
}

/* does (ka, ya) rank before (kb, yb): larger key first, then lower id */
static int before(float ka, int ya, float kb, int yb) { return ka > kb || (ka == kb && ya < yb); }

/* selection: mode A (k == 1) or top-k over all tokens (mode B) */
static int select_tokens(const Ctx *c, const float *x, const float *key32, int32_t *sel) {
  int V = c->V;
  if (c->mode == 0) {
    int a = 0;
    for (int y = 1; y < V; ++y)
      if (x[y] > x[a]) a = y;
    if (a == c->blank) {
      sel[0] = c->blank;
      return 1;
    }
    int best = -1;
    for (int y = 0; y < V; ++y) {
      if (y == c->blank) continue;
      if (best < 0 || before(key32[y], y, key32[best], best)) best = y;
    }
    sel[0] = best;
    return 1;
  }
  /* top-k by repeated selection of the best remaining token */
  for (int j = 0; j < c->k; ++j) {
    int best = -1;
    for (int y = 0; y < V; ++y) {
      int taken = 0;
      for (int i = 0; i < j; ++i) taken |= sel[i] == y;
      if (taken) continue;
      if (best < 0 || before(key32[y], y, key32[best], best)) best = y;
    }
    sel[j] = best;
  }
  return c->k;
}

/* ------------------------------------------------------------------------ */
/* step-wise entry: incoming states given as ids                              */
/* ------------------------------------------------------------------------ */
/* For each hypothesis h: selected tokens [H,k] (unused slots -1), reference
   fused scores [H,k] (fp64), next LM states [n_lm][H][k] and next phrase
   states [H,k]; optionally key32 [H,V], fused64 [H,V], lse64 [H].  lm_state is
   [n_lm][H].  Returns 0 or a negative code. */
int or_step_lms(const OrLM *const *lms, const float *lams, int n_lm, const OrTrie *tr,
                const float *logits, const int32_t *lm_state, const int32_t *boost_state, int H, int V,
                float beta, int blank, int k, int mode, float *key_out, double *fused_out,
                double *lse_out, int32_t *tokens, double *scores, int32_t *next_lm,
                int32_t *next_boost) {
  g_err[0] = 0;
  if (n_lm < 1 || n_lm > OR_MAXLM || !lms || !lams || H < 0 || k < 1 || k > V || k > 64 ||
      (mode == 0 && k != 1))
    return fail(OR_EARG, "bad step arguments");
  Ctx c;
  memset(&c, 0, sizeof c);
  for (int i = 0; i < n_lm; ++i) {
    if (!lms[i] || V != lms[i]->V || blank != lms[i]->blank) return fail(OR_EARG, "bad step arguments");
    c.lm[i] = lms[i];
    c.lam[i] = lams[i];
  }
  c.n_lm = n_lm;
  c.tr = tr;
  c.V = V;
  c.blank = blank;
  c.k = k;
  c.mode = mode;
  c.beta = beta;
  float *key = (float *)malloc((size_t)V * sizeof(float));
  double *f64 = (double *)malloc((size_t)V * sizeof(double));
  int64_t *nq = (int64_t *)malloc((size_t)V * sizeof(int64_t));
  int32_t sel[64];
  int32_t lmt[OR_MAXLM][OR_MAXN + 2];
  int32_t *lmp[OR_MAXLM];
  int lmlen[OR_MAXLM];
  for (int i = 0; i < OR_MAXLM; ++i) lmp[i] = lmt[i];
  int32_t *pt = (int32_t *)malloc((size_t)(tr ? tr->maxlen + 1 : 1) * sizeof(int32_t));
  int rc = OR_OK;
  for (int h = 0; h < H && rc == OR_OK; ++h) {
    for (int i = 0; i < n_lm; ++i) {
      lmlen[i] = or_lm_state_tuple(lms[i], lm_state[(int64_t)i * H + h], lmt[i]);
      if (lmlen[i] < 0 || (lmlen[i] == 1 && lmt[i][0] == blank)) rc = fail(OR_EARG, "invalid LM state");
    }
    if (rc != OR_OK) break;
    int plen = 0;
    if (tr) {
      plen = or_trie_node_tuple(tr, boost_state[h], pt);
      if (plen < 0) {
        rc = fail(OR_EARG, "invalid phrase state");
        break;
      }
    }
    const float *x = logits + (int64_t)h * V;
    double lse = score_row(&c, x, lmp, lmlen, pt, plen, key, f64, nq);
    if (key_out) memcpy(key_out + (int64_t)h * V, key, (size_t)V * sizeof(float));
    if (fused_out) memcpy(fused_out + (int64_t)h * V, f64, (size_t)V * sizeof(double));
    if (lse_out) lse_out[h] = lse;
    int ns = select_tokens(&c, x, key, sel);
    for (int j = 0; j < k; ++j) {
      int64_t o = (int64_t)h * k + j;
      int y = j < ns ? sel[j] : -1;
      tokens[o] = y;
      scores[o] = j < ns ? f64[y] : -INFINITY;
      next_boost[o] = (y < 0 || y == blank) ? boost_state[h] : (int32_t)nq[y];
      for (int i = 0; i < n_lm; ++i) {
        int64_t oi = (int64_t)i * H * k + o;
        if (y < 0 || y == blank) {
          next_lm[oi] = lm_state[(int64_t)i * H + h];
        } else {
          int32_t hist[OR_MAXN + 2];
          memcpy(hist, lmt[i], (size_t)lmlen[i] * sizeof(int32_t));
          hist[lmlen[i]] = y;
          next_lm[oi] = (int32_t)or_lm_state_of_history(lms[i], hist, lmlen[i] + 1);
        }
      }
    }
  }
  free(key);
  free(f64);
  free(nq);
  free(pt);
  return rc;
}

/* one LM: or_step_lms with n_lm = 1 and alpha_1 = lam */
int or_step(const OrLM *lm, const OrTrie *tr, const float *logits, const int32_t *lm_state,
            const int32_t *boost_state, int H, int V, float lam, float beta, int blank, int k,
            int mode, float *key_out, double *fused_out, double *lse_out, int32_t *tokens,
            double *scores, int32_t *next_lm, int32_t *next_boost) {
  return or_step_lms(&lm, &lam, 1, tr, logits, lm_state, boost_state, H, V, beta, blank, k, mode,
                     key_out, fused_out, lse_out, tokens, scores, next_lm, next_boost);
}

/* ------------------------------------------------------------------------ */
/* free-running decode over T frames from full histories                      */
/* ------------------------------------------------------------------------ */
typedef struct {
  int32_t *lm_hist[OR_MAXLM]; /* per LM: its initial state tuple + emitted tokens */
  int lm_len[OR_MAXLM];
  int32_t *ph_hist; /* phrase history (initial node tuple + emitted) */
  int ph_len;
  double score;
} Hyp;

typedef struct {
  const Ctx *c;
  const float *logits;
  int T, S, B, V;
  const int32_t *lm0, *q0; /* lm0: [n_lm][H] */
  const double *score0;
  int32_t *tokens, *parents; /* [T,H] */
  double *sel_score;         /* [T,H]: fused64 of the pick (B == 1) or the new score (B > 1) */
  int32_t *lm_out, *q_out; /* lm_out: [n_lm][H] */
  double *score_out;
  const int32_t *forced_tok, *forced_par; /* teacher forcing [T,H] or NULL */
  double tol;
  int64_t *near_ties, *mismatch_at; /* per stream */
  int s_begin, s_end;
  int rc;
} RunJob;

static void hyp_push(Hyp *h, int n_lm, int32_t y) {
  for (int i = 0; i < n_lm; ++i) h->lm_hist[i][h->lm_len[i]++] = y;
  h->ph_hist[h->ph_len++] = y;
}

/* do hypotheses pa + ya and pb + yb (blank appends nothing) hold the same
   history: the same LM histories (initial tuple and emitted tokens) for every
   LM and the same phrase history?  Compared token by token. */
static int same_history_after(const Hyp *pa, int32_t ya, const Hyp *pb, int32_t yb, int blank, int n_lm) {
  const int ea = ya != blank, eb = yb != blank;
  if (pa->ph_len + ea != pb->ph_len + eb) return 0;
  for (int i = 0; i < n_lm; ++i)
    if (pa->lm_len[i] + ea != pb->lm_len[i] + eb) return 0;
  for (int i = 0; i <= n_lm; ++i) {
    const int32_t *ha = i < n_lm ? pa->lm_hist[i] : pa->ph_hist;
    const int32_t *hb = i < n_lm ? pb->lm_hist[i] : pb->ph_hist;
    const int la = i < n_lm ? pa->lm_len[i] : pa->ph_len;
    const int lb = i < n_lm ? pb->lm_len[i] : pb->ph_len;
    for (int q = 0; q < la + ea; ++q) {
      const int32_t va = q < la ? ha[q] : ya, vb = q < lb ? hb[q] : yb;
      if (va != vb) return 0;
    }
  }
  return 1;
}

/* log(exp(a) + exp(b)) in fp64 */
static double log_add(double a, double b) {
  const double m = a > b ? a : b, d = a > b ? b - a : a - b;
  return m + log1p(exp(d));
}

static void hyp_copy(Hyp *d, const Hyp *p, int n_lm) {
  for (int i = 0; i < n_lm; ++i) {
    memcpy(d->lm_hist[i], p->lm_hist[i], (size_t)p->lm_len[i] * sizeof(int32_t));
    d->lm_len[i] = p->lm_len[i];
  }
  memcpy(d->ph_hist, p->ph_hist, (size_t)p->ph_len * sizeof(int32_t));
  d->ph_len = p->ph_len;
}

/* candidate of a beam step */
typedef struct {
  double score;
  int b, j;
  int32_t y;
} Cand;

static int cand_before(const Cand *a, const Cand *b) {
  if (a->score != b->score) return a->score > b->score;
  if (a->b != b->b) return a->b < b->b;
  return a->j < b->j;
}

static void *run_streams(void *arg) {
  RunJob *J = (RunJob *)arg;
  const Ctx *c = J->c;
  int V = J->V, B = J->B, T = J->T, k = c->k;
  int H = J->S * B;
  int cap = T + OR_MAXN + 8 + (c->tr ? c->tr->maxlen : 0);
  float *key = (float *)malloc((size_t)V * sizeof(float));
  double *f64 = (double *)malloc((size_t)V * sizeof(double));
  int64_t *nq = (int64_t *)malloc((size_t)V * sizeof(int64_t));
  Hyp *hy = (Hyp *)calloc((size_t)B, sizeof(Hyp));
  Hyp *nh = (Hyp *)calloc((size_t)B, sizeof(Hyp));
  Cand *cand = (Cand *)malloc((size_t)B * k * sizeof(Cand));
  int32_t *csel = (int32_t *)malloc((size_t)B * k * sizeof(int32_t));
  double *cf = (double *)malloc((size_t)B * k * sizeof(double));
  for (int b = 0; b < B; ++b) {
    for (int i = 0; i < c->n_lm; ++i) {
      hy[b].lm_hist[i] = (int32_t *)malloc((size_t)cap * sizeof(int32_t));
      nh[b].lm_hist[i] = (int32_t *)malloc((size_t)cap * sizeof(int32_t));
    }
    hy[b].ph_hist = (int32_t *)malloc((size_t)cap * sizeof(int32_t));
    nh[b].ph_hist = (int32_t *)malloc((size_t)cap * sizeof(int32_t));
  }
  for (int s = J->s_begin; s < J->s_end && J->rc == OR_OK; ++s) {
    for (int b = 0; b < B; ++b) {
      int h = s * B + b;
      Hyp *p = &hy[b];
      int bad = 0;
      for (int i = 0; i < c->n_lm; ++i) {
        p->lm_len[i] = or_lm_state_tuple(c->lm[i], J->lm0[(int64_t)i * H + h], p->lm_hist[i]);
        bad |= p->lm_len[i] < 0;
      }
      p->ph_len = c->tr ? or_trie_node_tuple(c->tr, J->q0[h], p->ph_hist) : 0;
      if (bad || p->ph_len < 0) {
        J->rc = OR_EARG;
        break;
      }
      p->score = B > 1 ? J->score0[h] : 0.0;
    }
    if (J->rc != OR_OK) break;
    for (int t = 0; t < T; ++t) {
      int nc = 0;
      for (int b = 0; b < B; ++b) {
        Hyp *p = &hy[b];
        if (B > 1 && p->score == -INFINITY) continue; /* dead hypotheses propose nothing */
        const float *x = J->logits + ((int64_t)t * H + s * B + b) * V;
        score_row(c, x, p->lm_hist, p->lm_len, p->ph_hist, p->ph_len, key, f64, nq);
        int ns = select_tokens(c, x, key, csel + b * k);
        for (int j = 0; j < ns; ++j) {
          int32_t y = csel[b * k + j];
          cand[nc].score = B > 1 ? p->score + f64[y] : f64[y];
          cand[nc].b = b;
          cand[nc].j = j;
          cand[nc].y = y;
          cf[b * k + j] = f64[y];
          ++nc;
        }
      }
      if (B == 1) {
        int h = s;
        int32_t y = cand[0].y;
        if (J->forced_tok && J->forced_tok[(int64_t)t * H + h] != y) {
          if (J->mismatch_at[s] < 0) J->mismatch_at[s] = t;
          y = J->forced_tok[(int64_t)t * H + h];
        }
        J->tokens[(int64_t)t * H + h] = y;
        if (J->sel_score) J->sel_score[(int64_t)t * H + h] = cand[0].score;
        if (y != c->blank) hyp_push(&hy[0], c->n_lm, y);
        continue;
      }
      /* recombination: candidates that reach the same history merge into the
         first of them in candidate order (parent asc, rank asc); its score is
         the log-sum of theirs, folded in that order */
      if (c->recombine) {
        int nr = 0;
        for (int q = 0; q < nc; ++q) {
          int r = -1;
          for (int u = 0; u < nr && r < 0; ++u)
            if (same_history_after(&hy[cand[u].b], cand[u].y, &hy[cand[q].b], cand[q].y, c->blank, c->n_lm)) r = u;
          if (r < 0) cand[nr++] = cand[q];
          else cand[r].score = log_add(cand[r].score, cand[q].score);
        }
        nc = nr;
      }
      /* beam: order candidates (score desc, parent asc, rank asc), keep B */
      for (int i = 1; i < nc; ++i) {
        Cand v = cand[i];
        int j = i - 1;
        while (j >= 0 && cand_before(&v, &cand[j])) {
          cand[j + 1] = cand[j];
          --j;
        }
        cand[j + 1] = v;
      }
      int keep = nc < B ? nc : B;
      /* teacher forcing: adopt the forced picks when they are distinct
         candidates, none of them is beaten by more than tol by a candidate
         they leave out, and their order agrees within tol */
      Cand pick[64];
      for (int i = 0; i < keep; ++i) pick[i] = cand[i];
      if (J->forced_tok) {
        int same = 1;
        for (int i = 0; i < B; ++i) {
          int64_t o = (int64_t)t * H + s * B + i;
          if (i < keep) same &= J->forced_par[o] == pick[i].b && J->forced_tok[o] == pick[i].y;
          else same &= J->forced_par[o] == -1;
        }
        if (!same) {
          int ok = 1;
          int idx[64];
          for (int i = 0; i < B && ok; ++i) {
            int64_t o = (int64_t)t * H + s * B + i;
            int fb = J->forced_par[o];
            int32_t fy = J->forced_tok[o];
            if (i >= keep) {
              ok = fb == -1;
              continue;
            }
            idx[i] = -1;
            for (int q = 0; q < nc; ++q)
              if (cand[q].b == fb && cand[q].y == fy) idx[i] = q;
            if (idx[i] < 0) ok = 0;
            for (int r = 0; r < i && ok; ++r)
              if (idx[r] == idx[i]) ok = 0;
          }
          if (ok) {
            double min_in = INFINITY, max_out = -INFINITY;
            for (int i = 0; i < keep; ++i)
              if (cand[idx[i]].score < min_in) min_in = cand[idx[i]].score;
            for (int q = 0; q < nc; ++q) {
              int in = 0;
              for (int i = 0; i < keep; ++i) in |= idx[i] == q;
              if (!in && cand[q].score > max_out) max_out = cand[q].score;
            }
            if (min_in < max_out - J->tol) ok = 0;
            for (int i = 0; i + 1 < keep && ok; ++i)
              if (cand[idx[i + 1]].score > cand[idx[i]].score + J->tol) ok = 0;
          }
          if (ok) {
            for (int i = 0; i < keep; ++i) pick[i] = cand[idx[i]];
            ++J->near_ties[s];
          } else if (J->mismatch_at[s] < 0) {
            J->mismatch_at[s] = t;
          }
        }
      }
      for (int i = 0; i < B; ++i) {
        int64_t o = (int64_t)t * H + s * B + i;
        Hyp *d = &nh[i];
        if (i < keep) {
          hyp_copy(d, &hy[pick[i].b], c->n_lm);
          d->score = pick[i].score;
          if (pick[i].y != c->blank) hyp_push(d, c->n_lm, pick[i].y);
          J->tokens[o] = pick[i].y;
          J->parents[o] = pick[i].b;
        } else {
          hyp_copy(d, &hy[i], c->n_lm); /* empty slot keeps its own history */
          d->score = -INFINITY;
          J->tokens[o] = -1;
          J->parents[o] = -1;
        }
        if (J->sel_score) J->sel_score[o] = d->score;
      }
      for (int i = 0; i < B; ++i) {
        Hyp tmp = hy[i];
        hy[i] = nh[i];
        nh[i] = tmp;
      }
    }
    for (int b = 0; b < B; ++b) {
      int h = s * B + b;
      Hyp *p = &hy[b];
      for (int i = 0; i < c->n_lm; ++i)
        J->lm_out[(int64_t)i * H + h] = (int32_t)or_lm_state_of_history(c->lm[i], p->lm_hist[i], p->lm_len[i]);
      J->q_out[h] = c->tr ? (int32_t)or_trie_state_of_history(c->tr, p->ph_hist, p->ph_len) : 0;
      if (J->score_out) J->score_out[h] = p->score;
    }
  }
  for (int b = 0; b < B; ++b) {
    for (int i = 0; i < c->n_lm; ++i) {
      free(hy[b].lm_hist[i]);
      free(nh[b].lm_hist[i]);
    }
    free(hy[b].ph_hist);
    free(nh[b].ph_hist);
  }
  free(hy);
  free(nh);
  free(cand);
  free(csel);
  free(cf);
  free(key);
  free(f64);
  free(nq);
  return NULL;
}

/* T frames, S streams of B hypotheses.  B == 1: greedy (k == 1).  B > 1: per
   hypothesis top-k, then per stream the best B of the B*k candidates by
   (score desc, parent asc, rank asc) with score = running score + fused64;
   slots left without a candidate are dead (score -inf, token/parent -1).
   forced_tok/forced_par (or NULL) replay a given decision sequence; a
   forced pick that is not within tol of the oracle's own choice is recorded
   in mismatch_at[s] (first frame, else -1); accepted near ties are counted.
   Threads split the streams. */
int or_run_lms(const OrLM *const *lms, const float *lams, int n_lm, const OrTrie *tr,
               const float *logits, int T, int S, int B, int V, int k, float beta, int blank,
               int mode, const int32_t *lm_state, const int32_t *boost_state,
               const double *hyp_score, int32_t *tokens, int32_t *parents, double *sel_score,
               int32_t *lm_out, int32_t *boost_out, double *score_out, const int32_t *forced_tok,
               const int32_t *forced_par, double tol, int64_t *near_ties, int64_t *mismatch_at,
               int n_threads, int recombine) {
  g_err[0] = 0;
  if (n_lm < 1 || n_lm > OR_MAXLM || !lms || !lams || T < 0 || S < 0 || B < 1 || B > 64 || k < 1 ||
      k > V || (B == 1 && k != 1) || (mode == 0 && k != 1) || (B > 1 && (!parents || !hyp_score)))
    return fail(OR_EARG, "bad run arguments");
  if (B * k > 4096) return fail(OR_EARG, "too many candidates");
  Ctx c;
  memset(&c, 0, sizeof c);
  for (int i = 0; i < n_lm; ++i) {
    if (!lms[i] || V != lms[i]->V || blank != lms[i]->blank) return fail(OR_EARG, "bad run arguments");
    c.lm[i] = lms[i];
    c.lam[i] = lams[i];
  }
  c.n_lm = n_lm;
  c.tr = tr;
  c.V = V;
  c.blank = blank;
  c.k = k;
  c.mode = mode;
  c.beta = beta;
  c.recombine = recombine != 0 && B > 1;
  if (n_threads < 1) n_threads = 1;
  if (n_threads > S) n_threads = S > 0 ? S : 1;
  for (int s = 0; s < S; ++s) {
    if (near_ties) near_ties[s] = 0;
    if (mismatch_at) mismatch_at[s] = -1;
  }
  int64_t *nt = near_ties ? near_ties : (int64_t *)calloc((size_t)S + 1, sizeof(int64_t));
  int64_t *mm = mismatch_at ? mismatch_at : (int64_t *)calloc((size_t)S + 1, sizeof(int64_t));
  if (!mismatch_at)
    for (int s = 0; s < S; ++s) mm[s] = -1;
  RunJob *jobs = (RunJob *)calloc((size_t)n_threads, sizeof(RunJob));
  pthread_t *th = (pthread_t *)calloc((size_t)n_threads, sizeof(pthread_t));
  for (int i = 0; i < n_threads; ++i) {
    RunJob *J = &jobs[i];
    J->c = &c;
    J->logits = logits;
    J->T = T;
    J->S = S;
    J->B = B;
    J->V = V;
    J->lm0 = lm_state;
    J->q0 = boost_state;
    J->score0 = hyp_score;
    J->tokens = tokens;
    J->parents = parents;
    J->sel_score = sel_score;
    J->lm_out = lm_out;
    J->q_out = boost_out;
    J->score_out = score_out;
    J->forced_tok = forced_tok;
    J->forced_par = forced_par;
    J->tol = tol;
    J->near_ties = nt;
    J->mismatch_at = mm;
    J->s_begin = (int)((int64_t)S * i / n_threads);
    J->s_end = (int)((int64_t)S * (i + 1) / n_threads);
    J->rc = OR_OK;
    if (n_threads > 1) pthread_create(&th[i], NULL, run_streams, J);
  }
  if (n_threads == 1) run_streams(&jobs[0]);
  else
    for (int i = 0; i < n_threads; ++i) pthread_join(th[i], NULL);
  int rc = OR_OK;
  for (int i = 0; i < n_threads; ++i)
    if (jobs[i].rc != OR_OK) rc = fail(jobs[i].rc, "invalid initial state");
  if (!near_ties) free(nt);
  if (!mismatch_at) free(mm);
  free(jobs);
  free(th);
  return rc;
}

/* one LM: or_run_lms with n_lm = 1 and alpha_1 = lam */
int or_run(const OrLM *lm, const OrTrie *tr, const float *logits, int T, int S, int B, int V,
           int k, float lam, float beta, int blank, int mode, const int32_t *lm_state,
           const int32_t *boost_state, const double *hyp_score, int32_t *tokens, int32_t *parents,
           double *sel_score, int32_t *lm_out, int32_t *boost_out, double *score_out,
           const int32_t *forced_tok, const int32_t *forced_par, double tol, int64_t *near_ties,
           int64_t *mismatch_at, int n_threads) {
  return or_run_lms(&lm, &lam, 1, tr, logits, T, S, B, V, k, beta, blank, mode, lm_state,
                    boost_state, hyp_score, tokens, parents, sel_score, lm_out, boost_out, score_out,
                    forced_tok, forced_par, tol, near_ties, mismatch_at, n_threads, 0);
}

/* ------------------------------------------------------------------------ */
/* end of stream: the LM terms of </s>                                        */
/* ------------------------------------------------------------------------ */
/* For each hypothesis h and LM i (in order): t_i = fl32(lam_i * lm_i(</s> |
   state)) with lm_i the fp32 backoff recursion; hyp_score[h] += t_i in fp64
   (in/out, or NULL), end_term[h] = (0 + t_1) + t_2 ... (or NULL).  lm_state is
   [n_lm][H].  A state that is blank or </s> is an error. */
int or_end_scores(const OrLM *const *lms, const float *lams, int n_lm, const int32_t *lm_state, int H,
                  double *hyp_score, double *end_term) {
  g_err[0] = 0;
  if (n_lm < 1 || n_lm > OR_MAXLM || !lms || !lams || H < 0) return fail(OR_EARG, "bad end arguments");
  for (int i = 0; i < n_lm; ++i)
    if (!lms[i]) return fail(OR_EARG, "bad end arguments");
  int32_t t[OR_MAXN + 2];
  for (int h = 0; h < H; ++h) {
    double term = 0.0;
    for (int i = 0; i < n_lm; ++i) {
      const OrLM *lm = lms[i];
      int len = or_lm_state_tuple(lm, lm_state[(int64_t)i * H + h], t);
      if (len < 0 || (len == 1 && (t[0] == lm->blank || t[0] == lm->V + 1)))
        return fail(OR_EARG, "invalid LM state");
      float v = or_lm_logp32(lm, t, len, lm->V + 1);
      float a = lams[i] * v;
      term = term + (double)a;
      if (hyp_score) hyp_score[h] = hyp_score[h] + (double)a;
    }
    if (end_term) end_term[h] = term;
  }
  return OR_OK;
}
