/*
 * TreeSpark draft-tree step: CPU ORACLE.  TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded fp64 implementation of what the draft-tree
 * hot path computes, written from the paper (arXiv 2609.22098):
 *   - parent-conditioned drafter conditional      (§1 Eq. 1; §3.2 item 1)
 *   - calibrated edge acceptance p-hat            (§3.4 Eq. 3)
 *   - best-first expansion with slots, caps, theta (§3.2 Algorithm 1; §3.5)
 *   - trees of many requests under one node budget (§4 per-request budgets)
 *   - without-replacement sibling draws at T>0    (§3.3 residual-proposal equation)
 *   - greedy verification by exact match          (§3.2 item 3; §3.3 first paragraph)
 *   - recursive rejection verification at T>0     (§3.3, Proposition 1)
 *   - the tree attention mask and position ids    (§3.2 item 3; §5)
 *
 * Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may load
 * this library.  It shares no code with the HIP path and the HIP path never
 * calls it.
 *
 * Readings where the paper is silent (each one is documented in the design notes):
 *   R1  randomness is Philox4x32-10 keyed by (seed) with counter
 *       (c0, path lo32, path hi32, request<<12 | depth<<4 | tag); a node is named
 *       by its structural path id (4 bits per level, digit = sibling index - 1),
 *       not by creation order.  Per-token draws: c0 = y>>2, word y&3.  Per-stage
 *       draws: c0 = j, word 0.  Tags: 1 expand, 2 accept, 3 bonus.
 *   R2  u = ((w>>9) + 0.5) * 2^-23: 24 significant bits, so the value is exact
 *       in fp32 as well as fp64; never 0 or 1 (it lies in [2^-24, 1 - 2^-24]).
 *   R3  the K sibling draws from the residual proposal q_T^(j) have two
 *       realisations (the distribution is the same):
 *       sampler 0, Gumbel-top-k over z/T + G(u_y): the order of the perturbed
 *         keys is a sequence of draws without replacement (Plackett-Luce);
 *       sampler 1, sequential draws as the paper states them: draw j picks a
 *         4096-token segment, then a 64-token block in it, then a token in
 *         it, each with probability proportional to its remaining q_T mass,
 *         from the three words of one Philox call (c0 = j, tag 4); at each
 *         level the pick is the first index whose cumulative mass exceeds
 *         u * (level total).
 *   R4  ties: top-k by (value desc, id asc); heap by (key desc, child depth asc,
 *       child path asc); argmax by smallest id.
 *   R5  expansion stops iff the popped key < log(theta) (strict); theta = 0 never stops.
 *   R6  N counts materialised nodes, root excluded; nodes at depth D get no slot.
 *   R7  a zero residual normaliser keeps the previous residual; acceptance is
 *       tested in the log domain: log u < log p_j(x) - log q_j(x).
 */
#define _GNU_SOURCE
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define TSO_TAG_EXPAND 1u
#define TSO_TAG_ACCEPT 2u
#define TSO_TAG_BONUS 3u
#define TSO_TAG_DRAW 4u

#define TSO_SEGMENT 4096 /* tokens per segment of the sequential sampler */
#define TSO_BLOCK 64     /* tokens per block */

/* ------------------------------------------------------------------------- */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as   */
/* easy as 1, 2, 3", SC'11): 10 rounds of a multiply-hi/lo bijection on four */
/* 32-bit counter words, with a Weyl-sequence key schedule.                  */
/* ------------------------------------------------------------------------- */
void tso_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k0 += 0x9E3779B9u; /* golden ratio */
      k1 += 0xBB67AE85u; /* sqrt(3) - 1   */
    }
    uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
    uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ c1 ^ k0;
    uint32_t n1 = lo1;
    uint32_t n2 = hi0 ^ c3 ^ k1;
    uint32_t n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* One 32-bit word of the node's stream (reading R1). */
static uint32_t draw_word(uint64_t seed, int request, int depth, uint64_t path,
                          uint32_t tag, uint32_t c0, int word) {
  uint32_t ctr[4], key[2], out[4];
  ctr[0] = c0;
  ctr[1] = (uint32_t)(path & 0xFFFFFFFFu);
  ctr[2] = (uint32_t)(path >> 32);
  ctr[3] = ((uint32_t)request << 12) | ((uint32_t)depth << 4) | tag;
  key[0] = (uint32_t)(seed & 0xFFFFFFFFu);
  key[1] = (uint32_t)(seed >> 32);
  tso_philox4x32_10(ctr, key, out);
  return out[word];
}

/* Reading R2: a uniform in (0,1) from the top 23 bits of a word. */
static double word_to_uniform(uint32_t w) {
  return ((double)(w >> 9) + 0.5) * (1.0 / 8388608.0);
}

double tso_u_token(uint64_t seed, int request, int depth, uint64_t path, int tag, int y) {
  return word_to_uniform(draw_word(seed, request, depth, path, (uint32_t)tag, (uint32_t)y >> 2, y & 3));
}

double tso_u_stage(uint64_t seed, int request, int depth, uint64_t path, int tag, int j) {
  return word_to_uniform(draw_word(seed, request, depth, path, (uint32_t)tag, (uint32_t)j, 0));
}

/* Standard Gumbel variate from a uniform: G = -log(-log u). */
static double gumbel(double u) { return -log(-log(u)); }

/* ------------------------------------------------------------------------- */
/* Calibrated edge acceptance, §3.4 Eq. 3: p-hat = sigmoid(a * logit(q0) + b). */
/* Returned as log p-hat from lq = log q0.                                    */
/* ------------------------------------------------------------------------- */

/* log(1 - exp(x)) for x <= 0, in the two-branch form of Maechler (2012). */
static double log1mexp(double x) {
  return (x > -M_LN2) ? log(-expm1(x)) : log1p(-exp(x));
}

double tso_log_phat(double lq, double a, double b) {
  double logit;
  if (lq >= 0.0)
    logit = INFINITY;                 /* q0 == 1 */
  else
    logit = lq - log1mexp(lq);        /* log q - log(1 - q) */
  double x = (a == 0.0) ? b : a * logit + b;
  if (x == INFINITY) return 0.0;
  if (x == -INFINITY) return -INFINITY;
  /* log sigmoid(x) */
  return (x >= 0.0) ? -log1p(exp(-x)) : x - log1p(exp(x));
}

/* ------------------------------------------------------------------------- */
/* Model tensors.  U [R][D][V] backbone logits (row d gives the logits of the  */
/* children of a depth-d parent, the LM-shifted block semantics of §3.1);      */
/* E [V][r] is W1 (row x = W1[x]); W2 [V][r] (row v = W2[v]), so that the      */
/* Markov bias is B(x, v) = <W1[x], W2[v]> (§3.1).                             */
/* ------------------------------------------------------------------------- */
typedef struct {
  int R, D, V, r;
  const float* U;
  const float* E;
  const float* W2;
} tso_model;

/* Smallest index among the not-yet-taken entries with the largest value. */
static int argmax_excluding(const double* v, int n, const unsigned char* taken) {
  int best = -1;
  for (int y = 0; y < n; ++y) {
    if (taken[y]) continue;
    if (best < 0 || v[y] > v[best]) best = y;
  }
  return best;
}

/* Take the first m of the order (value desc, id asc).  ids[m], vals[m]. */
static void top_m(const double* v, int n, int m, int* ids, double* vals, unsigned char* taken) {
  memset(taken, 0, (size_t)n);
  for (int i = 0; i < m; ++i) {
    int y = argmax_excluding(v, n, taken);
    ids[i] = y;
    vals[i] = (y >= 0) ? v[y] : -INFINITY;
    if (y >= 0) taken[y] = 1;
  }
}

static double logsumexp(const double* v, int n, double scale) {
  double m = -INFINITY;
  for (int y = 0; y < n; ++y)
    if (v[y] * scale > m) m = v[y] * scale;
  double s = 0.0;
  for (int y = 0; y < n; ++y) s += exp(v[y] * scale - m);
  return m + log(s);
}

/*
 * One node evaluation (§1 Eq. 1; Algorithm 1, definition of q0 and qT; §5.6):
 *   z[y]  = U[request][depth][y] + sum_i E[token][i] * W2[y][i]   (i ascending)
 *   lse0  = log sum_y exp(z[y]);  lseT = log sum_y exp(z[y] / T)  (T > 0)
 *   pi    = first K+1 tokens by (z desc, id asc)
 *   sigma = first K+1 tokens by (z/T + G(u_token(...expand...)) desc, id asc)   (T > 0)
 * Outputs with K+1 entries carry the first excluded value, for tie reporting.
 * z may be NULL.  Returns 0, or -1 on invalid arguments.
 */
/* One categorical pick: the first i in [0, n) whose cumulative mass exceeds
 * u * total.  gap: distance of the target to the nearest cumulative boundary,
 * relative to the total (for near-tie reporting). */
static int pick(const double* mass, int n, double u, double* gap) {
  double total = 0.0;
  for (int i = 0; i < n; ++i) total += mass[i];
  const double t = u * total;
  double c = 0.0;
  int chosen = -1;
  double lo = 0.0, hi = total;
  for (int i = 0; i < n; ++i) {
    if (!(mass[i] > 0.0)) continue;
    const double c1 = c + mass[i];
    if (c1 > t) { chosen = i; lo = c; hi = c1; break; }
    c = c1;
  }
  if (chosen < 0) /* rounding at the top end: the last index with mass */
    for (int i = n - 1; i >= 0 && chosen < 0; --i)
      if (mass[i] > 0.0) { chosen = i; lo = c - mass[i]; hi = c; }
  const double d = fmin(t - lo, hi - t) / total;
  if (d < *gap) *gap = d;
  return chosen;
}

/*
 * K draws without replacement from q_T (R3, sampler 1): §3.3's residual
 * proposal q_T^(j) = q_T restricted to the tokens not drawn before j, drawn
 * one after another.  Each draw picks a segment, a block in it and a token in
 * it, each in proportion to its remaining mass, which makes
 * P(token) = mass(token) / remaining mass.  gap[j - 1]: smallest relative gap
 * of the three picks of draw j.
 */
void tso_draw_sequential(const double* z, int V, double T, uint64_t seed, int request, int depth,
                         uint64_t path, int K, int32_t* sigma, double* gap) {
  const int nseg = (V + TSO_SEGMENT - 1) / TSO_SEGMENT;
  double* mass = (double*)malloc(sizeof(double) * (size_t)V);
  unsigned char* drawn = (unsigned char*)calloc((size_t)V, 1);
  double* seg = (double*)malloc(sizeof(double) * (size_t)nseg);
  double blk[TSO_SEGMENT / TSO_BLOCK];
  for (int j = 1; j <= K; ++j) {
    double* g = &gap[j - 1];
    *g = INFINITY;
    /* q_T^(j) up to its normaliser, relative to the largest remaining logit */
    double mx = -INFINITY;
    for (int y = 0; y < V; ++y)
      if (!drawn[y] && z[y] / T > mx) mx = z[y] / T;
    for (int y = 0; y < V; ++y) mass[y] = drawn[y] ? 0.0 : exp(z[y] / T - mx);
    uint32_t ctr[4] = {(uint32_t)j, (uint32_t)path, (uint32_t)(path >> 32),
                       ((uint32_t)request << 12) | ((uint32_t)depth << 4) | TSO_TAG_DRAW};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t w[4];
    tso_philox4x32_10(ctr, key, w);
    for (int sg = 0; sg < nseg; ++sg) {
      seg[sg] = 0.0;
      for (int y = sg * TSO_SEGMENT; y < V && y < (sg + 1) * TSO_SEGMENT; ++y) seg[sg] += mass[y];
    }
    const int sg = pick(seg, nseg, word_to_uniform(w[0]), g);
    if (sg < 0) {
      /* no mass left: every token with a finite logit is drawn, so this draw
       * and the ones after it are empty (q_T^(j) has no support) */
      for (int i = j; i <= K; ++i) { sigma[i - 1] = -1; gap[i - 1] = INFINITY; }
      break;
    }
    const int y0 = sg * TSO_SEGMENT;
    const int nb = ((V - y0 < TSO_SEGMENT ? V - y0 : TSO_SEGMENT) + TSO_BLOCK - 1) / TSO_BLOCK;
    for (int b = 0; b < nb; ++b) {
      blk[b] = 0.0;
      for (int y = y0 + b * TSO_BLOCK; y < V && y < y0 + (b + 1) * TSO_BLOCK; ++y) blk[b] += mass[y];
    }
    const int b = pick(blk, nb, word_to_uniform(w[1]), g);
    const int t0 = y0 + b * TSO_BLOCK;
    const int nt = V - t0 < TSO_BLOCK ? V - t0 : TSO_BLOCK;
    const int t = pick(mass + t0, nt, word_to_uniform(w[2]), g);
    sigma[j - 1] = t0 + t;
    drawn[t0 + t] = 1;
  }
  free(seg);
  free(drawn);
  free(mass);
}

/*
 * One node evaluation (§3.2 item 1; Algorithm 1): the conditional logits z,
 * lse0, lseT, the top K+1 by z (pi) and at T > 0 the K draws (sigma).
 * sigma_g: sampler 0, the K+1 largest Gumbel keys; sampler 1, sigma_g[j] is
 * the smallest relative gap of the picks of draw j + 1 (sigma_g[K] unused).
 */
int tso_eval(const tso_model* m, int request, int token, int depth, uint64_t path,
             double T, uint64_t seed, int sampler, int K,
             double* z_out, double* lse0, double* lseT,
             int* pi, double* pi_z, int* sigma, double* sigma_g, double* sigma_z) {
  if (!m || request < 0 || request >= m->R || token < 0 || token >= m->V || depth < 0 ||
      depth >= m->D || K < 1 || K > m->V || T < 0.0)
    return -1;
  const int V = m->V, r = m->r;
  double* z = z_out ? z_out : (double*)malloc(sizeof(double) * (size_t)V);
  unsigned char* taken = (unsigned char*)malloc((size_t)V);
  const float* urow = m->U + ((size_t)request * m->D + depth) * V;
  const float* e = m->E + (size_t)token * r;
  for (int y = 0; y < V; ++y) {
    double acc = 0.0;
    const float* w = m->W2 + (size_t)y * r;
    for (int i = 0; i < r; ++i) acc += (double)e[i] * (double)w[i];
    z[y] = (double)urow[y] + acc;
  }
  *lse0 = logsumexp(z, V, 1.0);
  int m1 = (K + 1 <= V) ? K + 1 : K;
  int* ids = (int*)malloc(sizeof(int) * (size_t)(K + 1));
  double* vals = (double*)malloc(sizeof(double) * (size_t)(K + 1));
  top_m(z, V, m1, ids, vals, taken);
  for (int i = 0; i < K; ++i) pi[i] = ids[i];
  if (pi_z) {
    for (int i = 0; i < m1; ++i) pi_z[i] = vals[i];
    if (m1 == K) pi_z[K] = -INFINITY;
  }
  if (T > 0.0 && sampler == 1) {
    *lseT = logsumexp(z, V, 1.0 / T);
    int32_t* sg = (int32_t*)malloc(sizeof(int32_t) * (size_t)K);
    double* gap = (double*)malloc(sizeof(double) * (size_t)K);
    tso_draw_sequential(z, V, T, seed, request, depth, path, K, sg, gap);
    for (int i = 0; i < K; ++i) {
      if (sigma) sigma[i] = sg[i];
      if (sigma_z) sigma_z[i] = sg[i] < 0 ? -INFINITY : z[sg[i]];
      if (sigma_g) sigma_g[i] = gap[i];
    }
    if (sigma_g) sigma_g[K] = NAN;
    free(gap);
    free(sg);
  } else if (T > 0.0) {
    *lseT = logsumexp(z, V, 1.0 / T);
    double* g = (double*)malloc(sizeof(double) * (size_t)V);
    for (int y = 0; y < V; ++y)
      g[y] = z[y] / T + gumbel(tso_u_token(seed, request, depth, path, TSO_TAG_EXPAND, y));
    top_m(g, V, m1, ids, vals, taken);
    for (int i = 0; i < K; ++i) {
      if (sigma) sigma[i] = ids[i];
      if (sigma_z) sigma_z[i] = z[ids[i]];
    }
    if (sigma_g) {
      for (int i = 0; i < m1; ++i) sigma_g[i] = vals[i];
      if (m1 == K) sigma_g[K] = -INFINITY;
    }
    free(g);
  } else {
    *lseT = NAN;
  }
  free(ids);
  free(vals);
  free(taken);
  if (!z_out) free(z);
  return 0;
}

/* ------------------------------------------------------------------------- */
/* Best-first tree expansion, §3.2 Algorithm 1 (one round), literally.        */
/* ------------------------------------------------------------------------- */
typedef struct {
  int n;            /* materialised nodes, root excluded */
  int evals;        /* node evaluations performed */
  int32_t* token;   /* [N+1], node 0 = root (anchor) */
  int32_t* parent;  /* -1 for the root */
  int32_t* depth;
  int32_t* rank;    /* sibling draw index j (1-based); 0 for the root */
  uint64_t* path;   /* structural path id (R1) */
  double* log_surv; /* log S(node) */
  double* log_q0;   /* log q0(token | parent) */
  double* log_qT;   /* log qT(token | parent), NaN at T = 0 */
  double* key;      /* key of the slot whose pop created the node */
  double* margin;   /* popped key minus the best key left in the heap (INFINITY if none) */
  double* eval_gap; /* smallest relative gap between consecutive sorted scores of the node's eval (top-k
                       logits; Gumbel keys), NaN if not evaluated */
  double* draw_gap; /* sequential draws: smallest gap of a pick to a cumulative boundary, relative to
                       the level's total (a mass, not a score); NaN otherwise or if not evaluated */
  double stop_key;  /* key of the slot that met the theta stop, NaN if none */
} tso_tree;

typedef struct {
  int K;
  double lse0, lseT;
  int* pi;
  double* pi_z;
  int* sigma;
  double* sigma_g;
  double* sigma_z;
} node_eval;

typedef struct {
  int v;            /* parent node index */
  int j;            /* 1-based sibling index of the child this slot creates */
  double key;
  int child_depth;
  uint64_t child_path;
} slot;

static double min_rel_gap(const double* vals, int n) {
  double g = INFINITY;
  for (int i = 0; i + 1 < n; ++i) {
    if (!isfinite(vals[i + 1])) continue;
    double d = (vals[i] - vals[i + 1]) / fmax(1.0, fabs(vals[i]));
    if (d < g) g = d;
  }
  return g;
}

static double min_of(const double* v, int n) {
  double m = INFINITY;
  for (int i = 0; i < n; ++i)
    if (v[i] < m) m = v[i];
  return m;
}

/* Token proposed by slot j of node v, its z, and the slot key (Algorithm 1; §3.3 pre-draw bound). */
static void slot_values(const node_eval* ev, double log_surv_v, int j, double T, int control_topk,
                        double a, double b, int* tok, double* zc, double* key) {
  if (T == 0.0 || control_topk) {
    /* Greedy: the best unused token under q0 is the j-th of pi. */
    *tok = ev->pi[j - 1];
    *zc = ev->pi_z[j - 1];
    *key = log_surv_v + tso_log_phat(*zc - ev->lse0, a, b);
  } else {
    /* Sampled: the j-th draw without replacement; the slot key is the admissible
     * pre-draw bound S(v) * p-hat(max q0 over tokens not drawn before j). */
    *tok = ev->sigma[j - 1];
    *zc = ev->sigma_z[j - 1];
    int bound = -1;
    double bound_z = 0.0;
    for (int i = 0; i < ev->K && bound < 0; ++i) {
      int used = 0;
      for (int s = 0; s < j - 1; ++s)
        if (ev->sigma[s] == ev->pi[i]) used = 1;
      if (!used) { bound = ev->pi[i]; bound_z = ev->pi_z[i]; }
    }
    *key = log_surv_v + tso_log_phat(bound_z - ev->lse0, a, b);
  }
}

static int slot_before(const slot* x, const slot* y) {
  if (x->key != y->key) return x->key > y->key;
  if (x->child_depth != y->child_depth) return x->child_depth < y->child_depth;
  return x->child_path < y->child_path;
}

/*
 * control_topk != 0 plants the biased control of §3.3 ("the failure mode"):
 * at T > 0 the children are the deterministic top-k of q0 instead of draws.
 */
int tso_expand_tree(const tso_model* m, int request, int anchor, double theta, int N, int K,
                    double a, double b, double T, uint64_t seed, int sampler, int control_topk,
                    tso_tree* out) {
  if (!m || !out || N < 0 || K < 1 || K > 16 || K > m->V || m->D > 16 || T < 0.0 ||
      theta < 0.0 || anchor < 0 || anchor >= m->V || request < 0 || request >= m->R)
    return -1;
  const double log_theta = (theta > 0.0) ? log(theta) : -INFINITY;
  node_eval* ev = (node_eval*)calloc((size_t)N + 1, sizeof(node_eval));
  slot* heap = (slot*)malloc(sizeof(slot) * ((size_t)N + 2));
  int nheap = 0;

  /* root: anchor token, depth 0, S = 1, path 0 */
  out->token[0] = anchor; out->parent[0] = -1; out->depth[0] = 0; out->rank[0] = 0;
  out->path[0] = 0; out->log_surv[0] = 0.0; out->log_q0[0] = 0.0; out->log_qT[0] = NAN;
  out->key[0] = 0.0; out->margin[0] = INFINITY;
  for (int i = 0; i <= N; ++i) out->eval_gap[i] = out->draw_gap[i] = NAN;
  out->stop_key = NAN;
  out->evals = 0;
  int n = 0;

#define EVALUATE(node)                                                                       \
  do {                                                                                       \
    node_eval* e_ = &ev[node];                                                               \
    e_->K = K;                                                                               \
    e_->pi = (int*)malloc(sizeof(int) * (size_t)K);                                          \
    e_->pi_z = (double*)malloc(sizeof(double) * (size_t)(K + 1));                            \
    e_->sigma = (int*)malloc(sizeof(int) * (size_t)K);                                       \
    e_->sigma_g = (double*)malloc(sizeof(double) * (size_t)(K + 1));                         \
    e_->sigma_z = (double*)malloc(sizeof(double) * (size_t)K);                               \
    tso_eval(m, request, out->token[node], out->depth[node], out->path[node], T, seed,       \
             sampler, K, NULL, &e_->lse0, &e_->lseT, e_->pi, e_->pi_z, e_->sigma,            \
             e_->sigma_g, e_->sigma_z);                                                      \
    double g_ = min_rel_gap(e_->pi_z, K + 1);                                                \
    if (T > 0.0 && sampler != 1) g_ = fmin(g_, min_rel_gap(e_->sigma_g, K + 1));             \
    out->eval_gap[node] = g_;                                                                \
    out->draw_gap[node] = (T > 0.0 && sampler == 1) ? min_of(e_->sigma_g, K) : NAN;          \
    out->evals++;                                                                            \
  } while (0)

  if (N > 0 && m->D > 0) {
    EVALUATE(0);
    slot s0;
    int tok; double zc;
    slot_values(&ev[0], 0.0, 1, T, control_topk, a, b, &tok, &zc, &s0.key);
    s0.v = 0; s0.j = 1; s0.child_depth = 1; s0.child_path = 0;
    heap[nheap++] = s0;
  }

  while (n < N && nheap > 0) {
    /* pop the best slot (plain scan: the heap is small) */
    int best = 0;
    for (int i = 1; i < nheap; ++i)
      if (slot_before(&heap[i], &heap[best])) best = i;
    slot s = heap[best];
    heap[best] = heap[--nheap];
    if (s.key < log_theta) { out->stop_key = s.key; break; }
    double next_best = -INFINITY;
    for (int i = 0; i < nheap; ++i)
      if (heap[i].key > next_best) next_best = heap[i].key;

    /* materialise the child */
    int v = s.v, j = s.j;
    int tok; double zc, key;
    slot_values(&ev[v], out->log_surv[v], j, T, control_topk, a, b, &tok, &zc, &key);
    int c = ++n;
    out->token[c] = tok;
    out->parent[c] = v;
    out->depth[c] = out->depth[v] + 1;
    out->rank[c] = j;
    out->path[c] = out->path[v] | ((uint64_t)(j - 1) << (4 * out->depth[v]));
    out->log_q0[c] = zc - ev[v].lse0;
    out->log_qT[c] = (T > 0.0) ? zc / T - ev[v].lseT : NAN;
    out->log_surv[c] = out->log_surv[v] + tso_log_phat(out->log_q0[c], a, b);
    out->key[c] = s.key;
    out->margin[c] = s.key - next_best;

    /* push slot(c) if it can have children; re-push slot(v) if v has < K children */
    if (out->depth[c] < m->D) {
      EVALUATE(c);
      slot sc;
      slot_values(&ev[c], out->log_surv[c], 1, T, control_topk, a, b, &tok, &zc, &sc.key);
      sc.v = c; sc.j = 1; sc.child_depth = out->depth[c] + 1; sc.child_path = out->path[c];
      heap[nheap++] = sc;
    }
    if (j < K) {
      slot sv;
      slot_values(&ev[v], out->log_surv[v], j + 1, T, control_topk, a, b, &tok, &zc, &sv.key);
      sv.v = v; sv.j = j + 1; sv.child_depth = out->depth[v] + 1;
      sv.child_path = out->path[v] | ((uint64_t)j << (4 * out->depth[v]));
      heap[nheap++] = sv;
    }
  }
#undef EVALUATE
  out->n = n;
  for (int i = 0; i <= N; ++i) {
    free(ev[i].pi); free(ev[i].pi_z); free(ev[i].sigma); free(ev[i].sigma_g); free(ev[i].sigma_z);
  }
  free(ev);
  free(heap);
  return 0;
}

/* ------------------------------------------------------------------------- */
/* Verification.                                                              */
/* target is [n+1][V]: row i holds the target's next-token logits after the  */
/* root path of node i (the row of node i under the tree attention mask).    */
/* ------------------------------------------------------------------------- */

/* Greedy verification by exact target-token match (§3.2 item 3; §3.3).
 * level_gap (optional, room for n + 1 values) receives, for each visited
 * node in walk order, the relative gap (best - second) / max(1, |best|) of
 * its target row: the decision taken there is unambiguous in fp32 unless
 * that gap is tiny. */
int tso_verify_greedy(const tso_tree* t, const float* target, int V, int32_t* path_nodes,
                      int32_t* path_len, int32_t* bonus, double* level_gap) {
  if (!t || !target || V < 1) return -1;
  int cur = 0, len = 0;
  for (;;) {
    const float* row = target + (size_t)cur * V;
    int g = 0;
    for (int y = 1; y < V; ++y)
      if (row[y] > row[g]) g = y;
    double second = -INFINITY;
    for (int y = 0; y < V; ++y)
      if (y != g && row[y] > second) second = row[y];
    double d = ((double)row[g] - second) / fmax(1.0, fabs((double)row[g]));
    if (level_gap) level_gap[len] = d;
    int next = -1;
    for (int c = 1; c <= t->n; ++c)
      if (t->parent[c] == cur && t->token[c] == g) { next = c; break; }
    if (next < 0) { *bonus = g; break; }
    path_nodes[len++] = next;
    cur = next;
  }
  *path_len = len;
  return 0;
}

/*
 * One node's recursive rejection stages with literal per-token vectors
 * (§3.3): q_j = norm(qT * 1[not drawn before j]); accept x_j with probability
 * min(1, p_j(x_j) / q_j(x_j)); after a rejection p_{j+1} = norm(max(p_j - q_j, 0)).
 * Runs all m stages as if every stage rejected (the values each stage sees when
 * it is reached).  ratio[j] = p_j(x_j)/q_j(x_j); Z[j] = sum max(p_j - q_j, 0).
 * p_final (optional) receives the residual after m rejections.
 */
int tso_residual_stages(int V, const double* p_in, const double* qT, int m, const int32_t* x,
                        double* ratio, double* Z, double* p_final) {
  double* p = (double*)malloc(sizeof(double) * (size_t)V);
  double* q = (double*)malloc(sizeof(double) * (size_t)V);
  unsigned char* drawn = (unsigned char*)calloc((size_t)V, 1);
  memcpy(p, p_in, sizeof(double) * (size_t)V);
  for (int j = 0; j < m; ++j) {
    double R = 0.0;
    for (int y = 0; y < V; ++y)
      if (!drawn[y]) R += qT[y];
    for (int y = 0; y < V; ++y) q[y] = drawn[y] ? 0.0 : qT[y] / R;
    ratio[j] = p[x[j]] / q[x[j]];
    double s = 0.0;
    for (int y = 0; y < V; ++y) {
      double d = p[y] - q[y];
      q[y] = d > 0.0 ? d : 0.0;
      s += q[y];
    }
    Z[j] = s;
    if (s > 0.0)
      for (int y = 0; y < V; ++y) p[y] = q[y] / s;
    drawn[x[j]] = 1;
  }
  if (p_final) memcpy(p_final, p, sizeof(double) * (size_t)V);
  free(p); free(q); free(drawn);
  return 0;
}

/*
 * Sampled verification (§3.3, Proposition 1; Algorithm 1 return line: each
 * visited parent's proposal is rebuilt from the logits and the draw order).
 * level_margin (optional, room for n + 1 values) receives, for each visited
 * node in walk order, the smallest relative margin of the decisions taken
 * there: |log u - log ratio| / max(1, |log ratio|) over its acceptance tests
 * and, at the last node, (best - second) / max(1, |best|) of the bonus keys.
 */
int tso_verify_sample(const tso_model* m, int request, const tso_tree* t, const float* target,
                      double T, uint64_t seed, int32_t* path_nodes, int32_t* path_len,
                      int32_t* bonus, double* level_margin) {
  if (!m || !t || !target || T <= 0.0) return -1;
  const int V = m->V;
  double* p = (double*)malloc(sizeof(double) * (size_t)V);
  double* qT = (double*)malloc(sizeof(double) * (size_t)V);
  double* q = (double*)malloc(sizeof(double) * (size_t)V);
  double* z = (double*)malloc(sizeof(double) * (size_t)V);
  unsigned char* drawn = (unsigned char*)malloc((size_t)V);
  int* kids = (int*)malloc(sizeof(int) * (size_t)(t->n + 1));
  int cur = 0, len = 0;
  for (;;) {
    double margin = INFINITY; /* of the decisions at this node */
    /* target residual starts at p = softmax(target row / T) */
    const float* row = target + (size_t)cur * V;
    double mx = -INFINITY;
    for (int y = 0; y < V; ++y)
      if ((double)row[y] / T > mx) mx = (double)row[y] / T;
    double s = 0.0;
    for (int y = 0; y < V; ++y) { p[y] = exp((double)row[y] / T - mx); s += p[y]; }
    for (int y = 0; y < V; ++y) p[y] /= s;

    int nk = 0;
    for (int c = 1; c <= t->n; ++c)
      if (t->parent[c] == cur) kids[nk++] = c; /* creation order = draw order */
    int accepted = -1;
    if (nk > 0) {
      double lse0, lseT;
      int* pi = (int*)malloc(sizeof(int) * 16);
      tso_eval(m, request, t->token[cur], t->depth[cur], t->path[cur], T, seed, 0, 1, z, &lse0,
               &lseT, pi, NULL, NULL, NULL, NULL);
      free(pi);
      for (int y = 0; y < V; ++y) qT[y] = exp(z[y] / T - lseT);
      memset(drawn, 0, (size_t)V);
      for (int j = 1; j <= nk && accepted < 0; ++j) {
        int x = t->token[kids[j - 1]];
        double R = 0.0;
        for (int y = 0; y < V; ++y)
          if (!drawn[y]) R += qT[y];
        for (int y = 0; y < V; ++y) q[y] = drawn[y] ? 0.0 : qT[y] / R;
        double u = tso_u_stage(seed, request, t->depth[cur], t->path[cur], TSO_TAG_ACCEPT, j);
        double log_ratio = log(p[x]) - ((z[x] / T - lseT) - log(R));
        double d = fabs(log(u) - log_ratio) / fmax(1.0, fabs(log_ratio));
        if (d < margin) margin = d;
        if (log(u) < log_ratio) {
          accepted = kids[j - 1];
        } else {
          double zs = 0.0;
          for (int y = 0; y < V; ++y) {
            double dd = p[y] - q[y];
            q[y] = dd > 0.0 ? dd : 0.0;
            zs += q[y];
          }
          if (zs > 0.0)
            for (int y = 0; y < V; ++y) p[y] = q[y] / zs;
          drawn[x] = 1;
        }
      }
    }
    if (accepted >= 0) {
      if (level_margin) level_margin[len] = margin;
      path_nodes[len++] = accepted;
      cur = accepted;
      continue;
    }
    /* bonus token: one draw from the final residual, as a Gumbel-max */
    int best = -1;
    double bk = -INFINITY, second = -INFINITY;
    for (int y = 0; y < V; ++y) {
      if (!(p[y] > 0.0)) continue;
      double k = log(p[y]) + gumbel(tso_u_token(seed, request, t->depth[cur], t->path[cur],
                                               TSO_TAG_BONUS, y));
      if (best < 0 || k > bk) { second = bk; bk = k; best = y; }
      else if (k > second) second = k;
    }
    double d = (bk - second) / fmax(1.0, fabs(bk));
    if (d < margin) margin = d;
    if (level_margin) level_margin[len] = margin;
    *bonus = best;
    break;
  }
  *path_len = len;
  free(p); free(qT); free(q); free(z); free(drawn); free(kids);
  return 0;
}

/* ------------------------------------------------------------------------- */
/* Tree attention mask and position ids for the target's verification pass   */
/* (§3.2 item 3: one forward over the flattened tree with a tree attention   */
/* mask and per-depth position ids; §5: an ancestor bitmask per row).        */
/* Row i (node 0 = the anchor) sees exactly the nodes on its root path,      */
/* itself included: bit j of row i is set iff j is i or an ancestor of i.    */
/* pos[i] = offset + depth(i), depth counted along the parent chain.         */
/* Rows n+1 .. cap-1 are zero and get pos -1.  W = ceil(cap / 32) words.     */
/* ------------------------------------------------------------------------- */
int tso_tree_mask(const int32_t* parent, int n, int cap, int offset, uint32_t* mask, int32_t* pos) {
  if (!parent || !mask || !pos || cap < 1 || n < 0 || n >= cap) return -1;
  const int W = (cap + 31) / 32;
  memset(mask, 0, sizeof(uint32_t) * (size_t)cap * W);
  for (int i = 0; i < cap; ++i) pos[i] = -1;
  for (int i = 0; i <= n; ++i) {
    int depth = 0;
    int a = i;
    for (;;) {
      mask[(size_t)i * W + (a >> 5)] |= 1u << (a & 31);
      if (a == 0) break;
      const int p = parent[a];
      if (p < 0 || p >= a) return -1; /* parents precede their children */
      a = p;
      ++depth;
    }
    pos[i] = offset + depth;
  }
  return 0;
}

/* ------------------------------------------------------------------------- */
/* Trees of R requests under one global node budget B (§4, per-request       */
/* budget allocation): one heap over every request's slots, popped by        */
/* (key desc, request asc, child depth asc, child path asc).  A popped slot  */
/* of request q is dropped if q already has N nodes or stopped; a key below  */
/* log(theta_q) stops q; otherwise the child is materialised in q's tree as  */
/* in Algorithm 1.  Expansion ends when B nodes exist in all (B <= 0: no     */
/* global budget) or the heap is empty.  trees[q] must hold N + 1 nodes.     */
/* ------------------------------------------------------------------------- */
typedef struct {
  int q, v, j;
  double key;
  int child_depth;
  uint64_t child_path;
} forest_slot;

static int forest_before(const forest_slot* x, const forest_slot* y) {
  if (x->key != y->key) return x->key > y->key;
  if (x->q != y->q) return x->q < y->q;
  if (x->child_depth != y->child_depth) return x->child_depth < y->child_depth;
  return x->child_path < y->child_path;
}

int tso_expand_forest(const tso_model* m, int R, const int32_t* anchor, const double* theta, int N,
                      int budget, int K, double a, double b, double T, uint64_t seed, int sampler,
                      tso_tree* trees) {
  if (!m || !anchor || !theta || !trees || R < 1 || R > m->R || N < 0 || K < 1 || K > 16 ||
      K > m->V || m->D > 16 || T < 0.0)
    return -1;
  node_eval** ev = (node_eval**)calloc((size_t)R, sizeof(node_eval*));
  forest_slot* heap = (forest_slot*)malloc(sizeof(forest_slot) * ((size_t)R * (2 * (size_t)N + 2)));
  int* done = (int*)calloc((size_t)R, sizeof(int));
  int nheap = 0, total = 0;
  for (int q = 0; q < R; ++q) {
    tso_tree* out = &trees[q];
    if (anchor[q] < 0 || anchor[q] >= m->V || theta[q] < 0.0) { free(ev); free(heap); free(done); return -1; }
    ev[q] = (node_eval*)calloc((size_t)N + 1, sizeof(node_eval));
    out->token[0] = anchor[q]; out->parent[0] = -1; out->depth[0] = 0; out->rank[0] = 0;
    out->path[0] = 0; out->log_surv[0] = 0.0; out->log_q0[0] = 0.0; out->log_qT[0] = NAN;
    out->key[0] = 0.0; out->margin[0] = INFINITY;
    for (int i = 0; i <= N; ++i) out->eval_gap[i] = out->draw_gap[i] = NAN;
    out->stop_key = NAN;
    out->evals = 0;
    out->n = 0;
  }

#define FOREST_EVAL(q, node)                                                                  \
  do {                                                                                       \
    node_eval* e_ = &ev[q][node];                                                            \
    tso_tree* t_ = &trees[q];                                                                \
    e_->K = K;                                                                               \
    e_->pi = (int*)malloc(sizeof(int) * (size_t)K);                                          \
    e_->pi_z = (double*)malloc(sizeof(double) * (size_t)(K + 1));                            \
    e_->sigma = (int*)malloc(sizeof(int) * (size_t)K);                                       \
    e_->sigma_g = (double*)malloc(sizeof(double) * (size_t)(K + 1));                         \
    e_->sigma_z = (double*)malloc(sizeof(double) * (size_t)K);                               \
    tso_eval(m, q, t_->token[node], t_->depth[node], t_->path[node], T, seed, sampler, K,     \
             NULL, &e_->lse0, &e_->lseT, e_->pi, e_->pi_z, e_->sigma, e_->sigma_g,           \
             e_->sigma_z);                                                                   \
    double g_ = min_rel_gap(e_->pi_z, K + 1);                                                \
    if (T > 0.0 && sampler != 1) g_ = fmin(g_, min_rel_gap(e_->sigma_g, K + 1));             \
    t_->eval_gap[node] = g_;                                                                 \
    t_->draw_gap[node] = (T > 0.0 && sampler == 1) ? min_of(e_->sigma_g, K) : NAN;           \
    t_->evals++;                                                                             \
  } while (0)

  if (N > 0 && m->D > 0) {
    for (int q = 0; q < R; ++q) {
      FOREST_EVAL(q, 0);
      forest_slot s0;
      int tok; double zc;
      slot_values(&ev[q][0], 0.0, 1, T, 0, a, b, &tok, &zc, &s0.key);
      s0.q = q; s0.v = 0; s0.j = 1; s0.child_depth = 1; s0.child_path = 0;
      heap[nheap++] = s0;
    }
  }
  while (nheap > 0 && (budget <= 0 || total < budget)) {
    int best = 0;
    for (int i = 1; i < nheap; ++i)
      if (forest_before(&heap[i], &heap[best])) best = i;
    forest_slot s = heap[best];
    heap[best] = heap[--nheap];
    const int q = s.q;
    tso_tree* out = &trees[q];
    if (done[q]) continue;
    const double log_theta = theta[q] > 0.0 ? log(theta[q]) : -INFINITY;
    if (s.key < log_theta) { done[q] = 1; out->stop_key = s.key; continue; }
    double next_best = -INFINITY;
    for (int i = 0; i < nheap; ++i)
      if (heap[i].q == q && heap[i].key > next_best) next_best = heap[i].key;
    const int v = s.v, j = s.j;
    int tok; double zc, key;
    slot_values(&ev[q][v], out->log_surv[v], j, T, 0, a, b, &tok, &zc, &key);
    const int c = ++out->n;
    ++total;
    out->token[c] = tok;
    out->parent[c] = v;
    out->depth[c] = out->depth[v] + 1;
    out->rank[c] = j;
    out->path[c] = out->path[v] | ((uint64_t)(j - 1) << (4 * out->depth[v]));
    out->log_q0[c] = zc - ev[q][v].lse0;
    out->log_qT[c] = (T > 0.0) ? zc / T - ev[q][v].lseT : NAN;
    out->log_surv[c] = out->log_surv[v] + tso_log_phat(out->log_q0[c], a, b);
    out->key[c] = s.key;
    out->margin[c] = s.key - next_best;
    if (out->n == N) { done[q] = 1; continue; }
    if (out->depth[c] < m->D) {
      FOREST_EVAL(q, c);
      forest_slot sc;
      slot_values(&ev[q][c], out->log_surv[c], 1, T, 0, a, b, &tok, &zc, &sc.key);
      sc.q = q; sc.v = c; sc.j = 1; sc.child_depth = out->depth[c] + 1; sc.child_path = out->path[c];
      heap[nheap++] = sc;
    }
    if (j < K) {
      forest_slot sv;
      slot_values(&ev[q][v], out->log_surv[v], j + 1, T, 0, a, b, &tok, &zc, &sv.key);
      sv.q = q; sv.v = v; sv.j = j + 1; sv.child_depth = out->depth[v] + 1;
      sv.child_path = out->path[v] | ((uint64_t)j << (4 * out->depth[v]));
      heap[nheap++] = sv;
    }
  }
#undef FOREST_EVAL
  for (int q = 0; q < R; ++q) {
    for (int i = 0; i <= N; ++i) {
      free(ev[q][i].pi); free(ev[q][i].pi_z); free(ev[q][i].sigma); free(ev[q][i].sigma_g);
      free(ev[q][i].sigma_z);
    }
    free(ev[q]);
  }
  free(ev);
  free(heap);
  free(done);
  return 0;
}
