/*
 * Plain CPU oracle for path-based TreeShap -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the tests, the package's smoke check and the benchmark's CPU-baseline
 * leg may load this library.  It shares no code, header, table or helper with
 * the GPU library; both sides are written independently from the paper
 * (Mitchell, Frank & Holmes, "GPUTreeShap", arXiv 2010.13972).
 *
 * Everything is fp64 and deliberately simple: no blocking, no fusion, no
 * reordering beyond what the cited definition or algorithm states.
 *
 * Routes (each must agree with the others before any GPU comparison):
 *   or_brute_shap / or_brute_interactions
 *       Eq. (2) and Eq. (3)-(6) by enumerating every feature subset, with the
 *       cover-weighted restriction f_S(x) of Section 2.1.  Small M only.
 *   or_treeshap
 *       Algorithm 1 (TreeShap: RECURSE / EXTEND / UNWIND) over every tree,
 *       OpenMP parallel over rows like the paper's CPU baseline (Section 4.2).
 *   or_interactions
 *       Section 2.2: TreeShap evaluated with feature j held present and held
 *       absent; phi_ij is half the difference, phi_ii from Eq. (6).
 *   or_path_brute
 *       Eq. (2) applied to the game of one merged path alone (one (row, path)
 *       pair), by subset enumeration; also its Eq. (3)-(6) counterpart.
 *   or_extract_paths
 *       Section 3.1-3.2: unique root-to-leaf paths, duplicates merged.
 *   or_pack_bfd, or_pack_ffd, or_pack_nf, or_pack_none
 *       Section 3.3 and Table 1: Best-Fit-Decreasing, First-Fit-Decreasing,
 *       Next-Fit and one-path-per-bin packing of path lengths.
 *
 * Readings of points the paper leaves open (each applied on both sides):
 *   - a split sends x left iff x < threshold (Section 3.1's half-open ranges),
 *     also inside Algorithm 1, whose printed test is x <= t;
 *   - a cover ratio r_child / r_parent with r_parent == 0 is taken as 0;
 *   - Algorithm 1 skips a subtree entered with zero_fraction == one_fraction
 *     == 0: every leaf below it has a path game that is identically zero, so
 *     it contributes nothing, and this keeps UNWIND's division by z finite;
 *   - the bias phi[M] is f_{empty set}(x), the cover-weighted expectation;
 *   - interaction outputs are (M+1) x (M+1) with the bias at [M][M].
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define OR_EXPORT __attribute__((visibility("default")))

/* ------------------------------------------------------------------------ */
/* ensemble view                                                            */
/* ------------------------------------------------------------------------ */

typedef struct {
  int32_t M, G;
  int64_t T;
  const int64_t *off;     /* [T+1] node offsets */
  const int32_t *group;   /* [T] */
  const int32_t *left, *right, *feat;
  const float *thr;
  const double *cover, *value;
} ens_t;

static ens_t make_ens(int32_t M, int32_t G, int64_t T, const int64_t *off,
                      const int32_t *group, const int32_t *left,
                      const int32_t *right, const int32_t *feat,
                      const float *thr, const double *cover,
                      const double *value) {
  ens_t e;
  e.M = M; e.G = G; e.T = T; e.off = off; e.group = group; e.left = left;
  e.right = right; e.feat = feat; e.thr = thr; e.cover = cover; e.value = value;
  return e;
}

/* cover ratio, with the zero-cover reading */
static double ratio(double child, double parent) {
  return parent > 0.0 ? child / parent : 0.0;
}

/* ------------------------------------------------------------------------ */
/* model output and the restriction f_S(x) (Section 2.1)                     */
/* ------------------------------------------------------------------------ */

static double tree_predict(const ens_t *e, int64_t t, const float *x) {
  const int64_t b = e->off[t];
  int32_t n = 0;
  while (e->left[b + n] >= 0) {
    int32_t d = e->feat[b + n];
    n = (x[d] < e->thr[b + n]) ? e->left[b + n] : e->right[b + n];
  }
  return e->value[b + n];
}

/* f_S(x) for one tree: follow x at splits on features in S, otherwise take
 * both children weighted by their share of the node's cover. */
static double tree_restrict(const ens_t *e, int64_t t, int32_t n,
                            const float *x, const unsigned char *in_S) {
  const int64_t b = e->off[t];
  if (e->left[b + n] < 0) return e->value[b + n];
  int32_t d = e->feat[b + n];
  int32_t a = e->left[b + n], c = e->right[b + n];
  if (in_S[d]) {
    return tree_restrict(e, t, (x[d] < e->thr[b + n]) ? a : c, x, in_S);
  }
  double r = e->cover[b + n];
  double wa = ratio(e->cover[b + a], r), wc = ratio(e->cover[b + c], r);
  double s = 0.0;
  if (wa != 0.0) s += wa * tree_restrict(e, t, a, x, in_S);
  if (wc != 0.0) s += wc * tree_restrict(e, t, c, x, in_S);
  return s;
}

OR_EXPORT void or_predict(int32_t M, int32_t G, int64_t T, const int64_t *off,
                          const int32_t *group, const int32_t *left,
                          const int32_t *right, const int32_t *feat,
                          const float *thr, const double *cover,
                          const double *value, const float *X, int64_t rows,
                          int64_t ld, double *out /* [rows, G] */) {
  ens_t e = make_ens(M, G, T, off, group, left, right, feat, thr, cover, value);
  for (int64_t r = 0; r < rows; r++) {
    for (int32_t g = 0; g < G; g++) out[r * G + g] = 0.0;
    for (int64_t t = 0; t < T; t++)
      out[r * G + e.group[t]] += tree_predict(&e, t, X + r * ld);
  }
}

/* expected value per group: f_{empty set}, independent of x */
OR_EXPORT void or_expected_value(int32_t M, int32_t G, int64_t T,
                                 const int64_t *off, const int32_t *group,
                                 const int32_t *left, const int32_t *right,
                                 const int32_t *feat, const float *thr,
                                 const double *cover, const double *value,
                                 double *out /* [G] */) {
  ens_t e = make_ens(M, G, T, off, group, left, right, feat, thr, cover, value);
  unsigned char *none = (unsigned char *)calloc((size_t)M + 1, 1);
  float *x = (float *)calloc((size_t)M + 1, sizeof(float));
  for (int32_t g = 0; g < G; g++) out[g] = 0.0;
  for (int64_t t = 0; t < T; t++)
    out[e.group[t]] += tree_restrict(&e, t, 0, x, none);
  free(none);
  free(x);
}

/* ------------------------------------------------------------------------ */
/* brute force: Eq. (2) and Eq. (3)-(6) over all 2^M subsets                 */
/* ------------------------------------------------------------------------ */

static double factorial(int n) {
  double f = 1.0;
  for (int i = 2; i <= n; i++) f *= (double)i;
  return f;
}

/* v[S] = sum over trees of group g of f_S(x), for every bitmask S */
static void all_restrictions(const ens_t *e, int32_t g, const float *x,
                             double *v) {
  const int32_t M = e->M;
  unsigned char *in_S = (unsigned char *)malloc((size_t)M);
  for (uint64_t S = 0; S < (1ull << M); S++) {
    for (int32_t i = 0; i < M; i++) in_S[i] = (unsigned char)((S >> i) & 1u);
    double s = 0.0;
    for (int64_t t = 0; t < e->T; t++)
      if (e->group[t] == g) s += tree_restrict(e, t, 0, x, in_S);
    v[S] = s;
  }
  free(in_S);
}

static int popcount64(uint64_t v) { return __builtin_popcountll(v); }

/* Shapley values of a game given as a table over bitmasks of n players:
 * phi_i = sum_{S not containing i} |S|!(n-|S|-1)!/n! [v(S+i) - v(S)]. */
static void shapley_from_table(int n, const double *v, double *phi) {
  const double nf = factorial(n);
  for (int i = 0; i < n; i++) {
    double s = 0.0;
    for (uint64_t S = 0; S < (1ull << n); S++) {
      if ((S >> i) & 1u) continue;
      int k = popcount64(S);
      double w = factorial(k) * factorial(n - k - 1) / nf;
      s += w * (v[S | (1ull << i)] - v[S]);
    }
    phi[i] = s;
  }
}

/* Shapley interaction index, Eq. (3)-(6), from a game table of n players.
 * out is n x n; diagonal from Eq. (6). */
static void interactions_from_table(int n, const double *v, double *out) {
  double *phi = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
  shapley_from_table(n, v, phi);
  const double denom = 2.0 * factorial(n - 1);
  for (int i = 0; i < n; i++) {
    for (int j = 0; j < n; j++) {
      if (i == j) continue;
      double s = 0.0;
      for (uint64_t S = 0; S < (1ull << n); S++) {
        if (((S >> i) & 1u) || ((S >> j) & 1u)) continue;
        int k = popcount64(S);
        double w = factorial(k) * factorial(n - k - 2) / denom;
        uint64_t Si = S | (1ull << i), Sj = S | (1ull << j);
        double nabla = v[Si | (1ull << j)] - v[Si] - v[Sj] + v[S];
        s += w * nabla;
      }
      out[i * n + j] = s;
    }
  }
  for (int i = 0; i < n; i++) {
    double s = phi[i];
    for (int j = 0; j < n; j++)
      if (j != i) s -= out[i * n + j];
    out[i * n + i] = s;
  }
  free(phi);
}

OR_EXPORT int or_brute_shap(int32_t M, int32_t G, int64_t T, const int64_t *off,
                            const int32_t *group, const int32_t *left,
                            const int32_t *right, const int32_t *feat,
                            const float *thr, const double *cover,
                            const double *value, const float *X, int64_t rows,
                            int64_t ld, double *phi /* [rows, G, M+1] */) {
  if (M > 20) return 1;
  ens_t e = make_ens(M, G, T, off, group, left, right, feat, thr, cover, value);
  double *v = (double *)malloc(sizeof(double) * ((size_t)1 << M));
  for (int64_t r = 0; r < rows; r++) {
    for (int32_t g = 0; g < G; g++) {
      double *out = phi + (r * G + g) * (M + 1);
      all_restrictions(&e, g, X + r * ld, v);
      shapley_from_table(M, v, out);
      out[M] = v[0];
    }
  }
  free(v);
  return 0;
}

OR_EXPORT int or_brute_interactions(
    int32_t M, int32_t G, int64_t T, const int64_t *off, const int32_t *group,
    const int32_t *left, const int32_t *right, const int32_t *feat,
    const float *thr, const double *cover, const double *value, const float *X,
    int64_t rows, int64_t ld, double *phi /* [rows, G, M+1, M+1] */) {
  if (M > 16 || M < 2) return 1;
  ens_t e = make_ens(M, G, T, off, group, left, right, feat, thr, cover, value);
  double *v = (double *)malloc(sizeof(double) * ((size_t)1 << M));
  double *blk = (double *)malloc(sizeof(double) * (size_t)M * M);
  const int64_t W = M + 1;
  for (int64_t r = 0; r < rows; r++) {
    for (int32_t g = 0; g < G; g++) {
      double *out = phi + (r * G + g) * W * W;
      memset(out, 0, sizeof(double) * (size_t)(W * W));
      all_restrictions(&e, g, X + r * ld, v);
      interactions_from_table(M, v, blk);
      for (int32_t i = 0; i < M; i++)
        for (int32_t j = 0; j < M; j++) out[i * W + j] = blk[i * M + j];
      out[M * W + M] = v[0];
    }
  }
  free(v);
  free(blk);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Algorithm 1: TreeShap (RECURSE / EXTEND / UNWIND), 0-based transcription  */
/* ------------------------------------------------------------------------ */

typedef struct {
  int32_t d;  /* feature, -1 for the initial dummy element */
  double z;   /* zero fraction */
  double o;   /* one fraction */
  double w;   /* permutation weight */
} pe_t;

/* EXTEND: append (p_i, p_z, p_o) to m[0..l-1] and update the weights. */
static void extend(pe_t *m, int l, double pz, double po, int32_t pi) {
  m[l].d = pi;
  m[l].z = pz;
  m[l].o = po;
  m[l].w = (l == 0) ? 1.0 : 0.0;
  for (int a = l - 1; a >= 0; a--) {
    m[a + 1].w += po * m[a].w * (double)(a + 1) / (double)(l + 1);
    m[a].w = pz * m[a].w * (double)(l - a) / (double)(l + 1);
  }
}

/* UNWIND element i out of m[0..l-1] in place; the result has l-1 elements. */
static void unwind(pe_t *m, int l, int i) {
  const double o = m[i].o, z = m[i].z;
  double n = m[l - 1].w;
  for (int j = l - 1; j >= 1; j--) { /* j is the 1-based position */
    pe_t *mj = &m[j - 1];
    if (o != 0.0) {
      double t = mj->w;
      mj->w = n * (double)l / ((double)j * o);
      n = t - mj->w * z * (double)(l - j) / (double)l;
    } else {
      mj->w = (mj->w * (double)l) / (z * (double)(l - j));
    }
  }
  for (int a = i; a < l - 1; a++) {
    m[a].d = m[a + 1].d;
    m[a].z = m[a + 1].z;
    m[a].o = m[a + 1].o;
  }
}

/* sum of the weights left after unwinding element i (a copy is unwound) */
static double unwound_sum(const pe_t *m, int l, int i, pe_t *tmp) {
  memcpy(tmp, m, sizeof(pe_t) * (size_t)l);
  unwind(tmp, l, i);
  double s = 0.0;
  for (int a = 0; a < l - 1; a++) s += tmp[a].w;
  return s;
}

typedef struct {
  const ens_t *e;
  int64_t t;
  const float *x;
  double *phi;     /* [M] */
  pe_t *stack;     /* (depth+2) levels x (depth+2) elements */
  int width;       /* elements per level */
  pe_t *tmp;
  int32_t cond;    /* conditioned feature, -1 for none */
  int cond_on;     /* 1: held present, 0: held absent */
} ts_ctx;

static void recurse(ts_ctx *c, int32_t j, int level, int l_parent, double pz,
                    double po, int32_t pi, double F) {
  const ens_t *e = c->e;
  const int64_t b = e->off[c->t];
  pe_t *m = c->stack + (size_t)level * c->width;
  int l = l_parent;
  if (level > 0)
    memcpy(m, c->stack + (size_t)(level - 1) * c->width,
           sizeof(pe_t) * (size_t)l_parent);
  if (!(c->cond >= 0 && pi == c->cond)) {
    extend(m, l, pz, po, pi);
    l += 1;
  }
  if (e->left[b + j] < 0) {
    const double v = e->value[b + j];
    for (int i = 1; i < l; i++) {
      double w = unwound_sum(m, l, i, c->tmp);
      c->phi[m[i].d] += F * w * (m[i].o - m[i].z) * v;
    }
    return;
  }
  const int32_t d = e->feat[b + j];
  const int32_t a = e->left[b + j], bb = e->right[b + j];
  const int go_left = c->x[d] < e->thr[b + j];
  const int32_t h = go_left ? a : bb, cold = go_left ? bb : a;
  const double rj = e->cover[b + j];
  if (c->cond >= 0 && d == c->cond) {
    /* the conditioned feature is never extended into the path */
    if (c->cond_on) {
      recurse(c, h, level + 1, l, 1.0, 1.0, d, F);
    } else {
      double Fh = F * ratio(e->cover[b + h], rj);
      double Fc = F * ratio(e->cover[b + cold], rj);
      if (Fh != 0.0) recurse(c, h, level + 1, l, 1.0, 1.0, d, Fh);
      if (Fc != 0.0) recurse(c, cold, level + 1, l, 1.0, 1.0, d, Fc);
    }
    return;
  }
  double iz = 1.0, io = 1.0;
  int k = -1;
  for (int a2 = 0; a2 < l; a2++)
    if (m[a2].d == d) { k = a2; break; }  /* FINDFIRST */
  if (k >= 0) {
    iz = m[k].z;
    io = m[k].o;
    unwind(m, l, k);
    l -= 1;
  }
  double zh = iz * e->cover[b + h], zc = iz * e->cover[b + cold];
  zh = rj > 0.0 ? zh / rj : 0.0;
  zc = rj > 0.0 ? zc / rj : 0.0;
  if (!(zh == 0.0 && io == 0.0)) recurse(c, h, level + 1, l, zh, io, d, F);
  if (zc != 0.0) recurse(c, cold, level + 1, l, zc, 0.0, d, F);
}

static int tree_depth(const ens_t *e, int64_t t) {
  const int64_t b = e->off[t];
  const int32_t n = (int32_t)(e->off[t + 1] - b);
  int *dep = (int *)calloc((size_t)n, sizeof(int));
  int best = 0;
  /* nodes may be stored in any order: iterate to a fixed point */
  int changed = 1;
  while (changed) {
    changed = 0;
    for (int32_t i = 0; i < n; i++) {
      if (e->left[b + i] < 0) continue;
      int32_t ch[2] = {e->left[b + i], e->right[b + i]};
      for (int q = 0; q < 2; q++)
        if (dep[ch[q]] < dep[i] + 1) { dep[ch[q]] = dep[i] + 1; changed = 1; }
    }
  }
  for (int32_t i = 0; i < n; i++) best = dep[i] > best ? dep[i] : best;
  free(dep);
  return best;
}

static int ensemble_depth(const ens_t *e) {
  int D = 0;
  for (int64_t t = 0; t < e->T; t++) {
    int d = tree_depth(e, t);
    D = d > D ? d : D;
  }
  return D;
}

/* phi_acc[M] += TreeShap of tree t (Algorithm 1), optionally conditioned */
static void treeshap_tree(const ens_t *e, int64_t t, const float *x, double *phi,
                          pe_t *stack, int width, pe_t *tmp, int32_t cond,
                          int cond_on) {
  ts_ctx c;
  c.e = e; c.t = t; c.x = x; c.phi = phi; c.stack = stack; c.width = width;
  c.tmp = tmp; c.cond = cond; c.cond_on = cond_on;
  recurse(&c, 0, 0, 0, 1.0, 1.0, -1, 1.0);
}

OR_EXPORT int or_treeshap(int32_t M, int32_t G, int64_t T, const int64_t *off,
                          const int32_t *group, const int32_t *left,
                          const int32_t *right, const int32_t *feat,
                          const float *thr, const double *cover,
                          const double *value, const float *X, int64_t rows,
                          int64_t ld, double *phi /* [rows, G, M+1] */,
                          int32_t nthreads) {
  ens_t e = make_ens(M, G, T, off, group, left, right, feat, thr, cover, value);
  const int D = ensemble_depth(&e);
  const int width = D + 2;
  double *bias = (double *)calloc((size_t)G, sizeof(double));
  or_expected_value(M, G, T, off, group, left, right, feat, thr, cover, value,
                    bias);
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
#pragma omp parallel
  {
    pe_t *stack = (pe_t *)malloc(sizeof(pe_t) * (size_t)width * (width + 1));
    pe_t *tmp = (pe_t *)malloc(sizeof(pe_t) * (size_t)width);
    double *acc = (double *)malloc(sizeof(double) * (size_t)M);
#pragma omp for schedule(dynamic, 1)
    for (int64_t r = 0; r < rows; r++) {
      for (int32_t g = 0; g < G; g++) {
        memset(acc, 0, sizeof(double) * (size_t)M);
        for (int64_t t = 0; t < T; t++)
          if (e.group[t] == g)
            treeshap_tree(&e, t, X + r * ld, acc, stack, width, tmp, -1, 0);
        double *out = phi + (r * G + g) * (M + 1);
        for (int32_t i = 0; i < M; i++) out[i] = acc[i];
        out[M] = bias[g];
      }
    }
    free(stack);
    free(tmp);
    free(acc);
  }
  free(bias);
  return 0;
}

static int tree_uses_feature(const ens_t *e, int64_t t, int32_t j) {
  for (int64_t n = e->off[t]; n < e->off[t + 1]; n++)
    if (e->left[n] >= 0 && e->feat[n] == j) return 1;
  return 0;
}

/* Section 2.2: interaction values by conditioning.  For every feature j,
 * TreeShap runs with j held present and held absent (j never extended);
 * phi_ij = (phi_i|j present - phi_i|j absent) / 2 for i != j, and
 * phi_ii = phi_i - sum_{j != i} phi_ij (Eq. 6).  A tree that never splits on
 * j gives identical present/absent runs, so it is skipped for that j. */
OR_EXPORT int or_interactions(int32_t M, int32_t G, int64_t T,
                              const int64_t *off, const int32_t *group,
                              const int32_t *left, const int32_t *right,
                              const int32_t *feat, const float *thr,
                              const double *cover, const double *value,
                              const float *X, int64_t rows, int64_t ld,
                              double *phi /* [rows, G, M+1, M+1] */,
                              int32_t nthreads) {
  ens_t e = make_ens(M, G, T, off, group, left, right, feat, thr, cover, value);
  const int D = ensemble_depth(&e);
  const int width = D + 2;
  const int64_t W = M + 1;
  double *bias = (double *)calloc((size_t)G, sizeof(double));
  or_expected_value(M, G, T, off, group, left, right, feat, thr, cover, value,
                    bias);
  unsigned char *uses = (unsigned char *)malloc((size_t)T * (size_t)M);
  for (int64_t t = 0; t < T; t++)
    for (int32_t j = 0; j < M; j++) uses[t * M + j] = (unsigned char)tree_uses_feature(&e, t, j);
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
#pragma omp parallel
  {
    pe_t *stack = (pe_t *)malloc(sizeof(pe_t) * (size_t)width * (width + 1));
    pe_t *tmp = (pe_t *)malloc(sizeof(pe_t) * (size_t)width);
    double *plain = (double *)malloc(sizeof(double) * (size_t)M);
    double *on = (double *)malloc(sizeof(double) * (size_t)M);
    double *offv = (double *)malloc(sizeof(double) * (size_t)M);
#pragma omp for schedule(dynamic, 1)
    for (int64_t r = 0; r < rows; r++) {
      const float *x = X + r * ld;
      for (int32_t g = 0; g < G; g++) {
        double *out = phi + (r * G + g) * W * W;
        memset(out, 0, sizeof(double) * (size_t)(W * W));
        memset(plain, 0, sizeof(double) * (size_t)M);
        for (int64_t t = 0; t < T; t++)
          if (e.group[t] == g)
            treeshap_tree(&e, t, x, plain, stack, width, tmp, -1, 0);
        for (int32_t j = 0; j < M; j++) {
          memset(on, 0, sizeof(double) * (size_t)M);
          memset(offv, 0, sizeof(double) * (size_t)M);
          for (int64_t t = 0; t < T; t++) {
            if (e.group[t] != g || !uses[t * M + j]) continue;
            treeshap_tree(&e, t, x, on, stack, width, tmp, j, 1);
            treeshap_tree(&e, t, x, offv, stack, width, tmp, j, 0);
          }
          for (int32_t i = 0; i < M; i++)
            if (i != j) out[i * W + j] = (on[i] - offv[i]) / 2.0;
        }
        for (int32_t i = 0; i < M; i++) {
          double s = plain[i];
          for (int32_t j = 0; j < M; j++)
            if (j != i) s -= out[i * W + j];
          out[i * W + i] = s;
        }
        out[M * W + M] = bias[g];
      }
    }
    free(stack); free(tmp); free(plain); free(on); free(offv);
  }
  free(uses);
  free(bias);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* one merged path on its own: Eq. (2) and Eq. (3)-(6) by enumeration        */
/* ------------------------------------------------------------------------ */

/* The game of a single path with features k = 0..q-1 (root excluded):
 * v(S) = v * prod_{k in S} o_k * prod_{k not in S} z_k, where o_k tests
 * lower_k <= x < upper_k.  Output phi_out[q] (Shapley value per element) and,
 * when inter_out != NULL, the q x q interaction matrix (Eq. 3-6). */
OR_EXPORT int or_path_brute(int32_t q, const int32_t *feature,
                            const float *lower, const float *upper,
                            const double *zero_fraction, double v,
                            const float *x, double *phi_out,
                            double *inter_out) {
  if (q < 0 || q > 20) return 1;
  if (q == 0) return 0;
  double *o = (double *)malloc(sizeof(double) * (size_t)q);
  for (int k = 0; k < q; k++) {
    float xv = x[feature[k]];
    o[k] = (xv >= lower[k] && xv < upper[k]) ? 1.0 : 0.0;
  }
  double *game = (double *)malloc(sizeof(double) * ((size_t)1 << q));
  for (uint64_t S = 0; S < (1ull << q); S++) {
    double p = v;
    for (int k = 0; k < q; k++) p *= ((S >> k) & 1u) ? o[k] : zero_fraction[k];
    game[S] = p;
  }
  shapley_from_table(q, game, phi_out);
  if (inter_out != NULL) {
    if (q == 1) inter_out[0] = phi_out[0];
    else interactions_from_table(q, game, inter_out);
  }
  free(game);
  free(o);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Section 3.1-3.2: unique paths with duplicate features merged              */
/* ------------------------------------------------------------------------ */
/*
 * Canonical output order: trees in input order; within a tree, leaves in
 * depth-first preorder with the left child (x < t) first; path_idx counts up
 * from 0 over the whole ensemble.  Each path is its root element (feature
 * -1, range (-inf, +inf), zero fraction 1, the leaf value) followed by one
 * element per distinct split feature in ascending feature order.  A left
 * turn at threshold t bounds the range above by t, a right turn below by t;
 * repeats of a feature intersect the ranges and multiply zero fractions in
 * root-to-leaf order.  The bias term of a path is v * (1 * z_1 * z_2 * ...)
 * in element order; each tree sums its paths' terms in path order, and
 * bias[g] sums the trees of group g in tree order.
 */

typedef struct {
  int32_t feat;
  float lo, hi;
  double z;
} raw_t;

static int cmp_raw_feat(const void *a, const void *b) {
  const raw_t *x = (const raw_t *)a, *y = (const raw_t *)b;
  return (x->feat > y->feat) - (x->feat < y->feat);
}

typedef struct {
  int64_t *path_idx;
  int32_t *feature, *group;
  float *lower, *upper;
  double *zero, *v;
  int64_t cap, n, paths;
  double *bias;
  double tree_sum; /* the current tree's bias terms so far */
} out_t;

static void emit_leaf(const ens_t *e, int64_t t, int32_t leaf, raw_t *splits,
                      int ns, out_t *o) {
  const int64_t b = e->off[t];
  const double v = e->value[b + leaf];
  const int32_t g = e->group[t];
  /* stable insertion sort by feature keeps root-to-leaf order among repeats */
  raw_t *s = (raw_t *)malloc(sizeof(raw_t) * (size_t)(ns > 0 ? ns : 1));
  memcpy(s, splits, sizeof(raw_t) * (size_t)ns);
  for (int i = 1; i < ns; i++) {
    raw_t key = s[i];
    int j = i - 1;
    while (j >= 0 && cmp_raw_feat(&s[j], &key) > 0) { s[j + 1] = s[j]; j--; }
    s[j + 1] = key;
  }
  /* merged elements */
  int nm = 0;
  raw_t *m = (raw_t *)malloc(sizeof(raw_t) * (size_t)(ns > 0 ? ns : 1));
  for (int i = 0; i < ns; i++) {
    if (nm > 0 && m[nm - 1].feat == s[i].feat) {
      if (s[i].lo > m[nm - 1].lo) m[nm - 1].lo = s[i].lo;
      if (s[i].hi < m[nm - 1].hi) m[nm - 1].hi = s[i].hi;
      m[nm - 1].z = m[nm - 1].z * s[i].z;
    } else {
      m[nm].feat = s[i].feat;
      m[nm].lo = s[i].lo;
      m[nm].hi = s[i].hi;
      m[nm].z = 1.0 * s[i].z;
      nm++;
    }
  }
  double prod = 1.0;
  for (int i = 0; i < nm; i++) prod = prod * m[i].z;
  o->tree_sum = o->tree_sum + v * prod;
  for (int i = -1; i < nm; i++) {
    if (o->n < o->cap) {
      int64_t k = o->n;
      o->path_idx[k] = o->paths;
      o->group[k] = g;
      o->v[k] = v;
      if (i < 0) {
        o->feature[k] = -1;
        o->lower[k] = -INFINITY;
        o->upper[k] = INFINITY;
        o->zero[k] = 1.0;
      } else {
        o->feature[k] = m[i].feat;
        o->lower[k] = m[i].lo;
        o->upper[k] = m[i].hi;
        o->zero[k] = m[i].z;
      }
    }
    o->n++;
  }
  o->paths++;
  free(m);
  free(s);
}

static void walk(const ens_t *e, int64_t t, int32_t n, raw_t *splits, int ns,
                 out_t *o) {
  const int64_t b = e->off[t];
  if (e->left[b + n] < 0) {
    emit_leaf(e, t, n, splits, ns, o);
    return;
  }
  const int32_t d = e->feat[b + n];
  const float th = e->thr[b + n];
  const double r = e->cover[b + n];
  const int32_t a = e->left[b + n], c = e->right[b + n];
  splits[ns].feat = d;
  splits[ns].lo = -INFINITY;
  splits[ns].hi = th;
  splits[ns].z = ratio(e->cover[b + a], r);
  walk(e, t, a, splits, ns + 1, o);
  splits[ns].feat = d;
  splits[ns].lo = th;
  splits[ns].hi = INFINITY;
  splits[ns].z = ratio(e->cover[b + c], r);
  walk(e, t, c, splits, ns + 1, o);
}

/* Returns the element count; writes up to cap elements.  *num_paths gets the
 * path count; bias (may be NULL) is [G] and is overwritten. */
OR_EXPORT int64_t or_extract_paths(
    int32_t M, int32_t G, int64_t T, const int64_t *off, const int32_t *group,
    const int32_t *left, const int32_t *right, const int32_t *feat,
    const float *thr, const double *cover, const double *value, int64_t cap,
    int64_t *path_idx, int32_t *feature, int32_t *egroup, float *lower,
    float *upper, double *zero, double *v, int64_t *num_paths, double *bias) {
  ens_t e = make_ens(M, G, T, off, group, left, right, feat, thr, cover, value);
  out_t o;
  o.path_idx = path_idx; o.feature = feature; o.group = egroup; o.lower = lower;
  o.upper = upper; o.zero = zero; o.v = v; o.cap = cap; o.n = 0; o.paths = 0;
  o.bias = bias;
  if (bias)
    for (int32_t g = 0; g < G; g++) bias[g] = 0.0;
  const int D = ensemble_depth(&e);
  raw_t *splits = (raw_t *)malloc(sizeof(raw_t) * (size_t)(D + 1));
  for (int64_t t = 0; t < T; t++) {
    o.tree_sum = 0.0;
    walk(&e, t, 0, splits, 0, &o);
    if (bias) bias[group[t]] = bias[group[t]] + o.tree_sum;
  }
  free(splits);
  *num_paths = o.paths;
  return o.n;
}

/* ------------------------------------------------------------------------ */
/* Section 3.3: Best-Fit-Decreasing                                          */
/* ------------------------------------------------------------------------ */
/*
 * Items are paths with size = path length (root included).  Each group is
 * packed on its own, groups in ascending order, bins numbered in opening
 * order across the whole run.  Items are taken by non-increasing size, ties
 * by ascending path index; each goes to the open bin of its group with the
 * smallest residual capacity that still holds it (ties: lowest bin number),
 * else to a new bin.  A bin may be filled exactly to capacity.
 * Outputs: bin_of[p], lane_of[p] (offset of the path inside its bin, in
 * placement order).  Returns the number of bins, or -1 if an item exceeds
 * the capacity.
 */
typedef struct {
  int32_t size;
  int32_t group;
  int64_t idx;
} item_t;

static int cmp_item(const void *a, const void *b) {
  const item_t *x = (const item_t *)a, *y = (const item_t *)b;
  if (x->group != y->group) return (x->group > y->group) - (x->group < y->group);
  if (x->size != y->size) return (x->size < y->size) - (x->size > y->size);
  return (x->idx > y->idx) - (x->idx < y->idx);
}

OR_EXPORT int64_t or_pack_bfd(int64_t n, const int32_t *size,
                              const int32_t *group, int32_t capacity,
                              int64_t *bin_of, int32_t *lane_of) {
  item_t *it = (item_t *)malloc(sizeof(item_t) * (size_t)(n > 0 ? n : 1));
  for (int64_t p = 0; p < n; p++) {
    if (size[p] < 1 || size[p] > capacity) { free(it); return -1; }
    it[p].size = size[p];
    it[p].group = group[p];
    it[p].idx = p;
  }
  qsort(it, (size_t)n, sizeof(item_t), cmp_item);
  int32_t *resid = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
  int64_t nbins = 0, group_first_bin = 0;
  int32_t cur_group = n > 0 ? it[0].group : 0;
  for (int64_t k = 0; k < n; k++) {
    if (it[k].group != cur_group) {
      cur_group = it[k].group;
      group_first_bin = nbins;
    }
    const int32_t s = it[k].size;
    int64_t best = -1;
    for (int64_t b = group_first_bin; b < nbins; b++) {
      if (resid[b] < s) continue;
      if (best < 0 || resid[b] < resid[best]) best = b;
      if (resid[b] == s) break; /* cannot do better; first such bin is lowest */
    }
    if (best < 0) {
      best = nbins++;
      resid[best] = capacity;
    }
    bin_of[it[k].idx] = best;
    lane_of[it[k].idx] = capacity - resid[best];
    resid[best] -= s;
  }
  free(resid);
  free(it);
  return nbins;
}

/* ------------------------------------------------------------------------ */
/* Section 3.3 / Table 1: the other packing heuristics                       */
/* ------------------------------------------------------------------------ */
/*
 * First-Fit-Decreasing: the processing order of or_pack_bfd (by group, then
 * non-increasing size, then ascending path index); each item goes to the
 * lowest-numbered open bin of its group that still holds it, else a new bin.
 * Same outputs and return value as or_pack_bfd.
 */
OR_EXPORT int64_t or_pack_ffd(int64_t n, const int32_t *size,
                              const int32_t *group, int32_t capacity,
                              int64_t *bin_of, int32_t *lane_of) {
  item_t *it = (item_t *)malloc(sizeof(item_t) * (size_t)(n > 0 ? n : 1));
  for (int64_t p = 0; p < n; p++) {
    if (size[p] < 1 || size[p] > capacity) { free(it); return -1; }
    it[p].size = size[p];
    it[p].group = group[p];
    it[p].idx = p;
  }
  qsort(it, (size_t)n, sizeof(item_t), cmp_item);
  int32_t *resid = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
  int64_t nbins = 0, group_first_bin = 0;
  int32_t cur_group = n > 0 ? it[0].group : 0;
  for (int64_t k = 0; k < n; k++) {
    if (it[k].group != cur_group) {
      cur_group = it[k].group;
      group_first_bin = nbins;
    }
    const int32_t s = it[k].size;
    int64_t first = -1;
    for (int64_t b = group_first_bin; b < nbins; b++) {
      if (resid[b] >= s) { first = b; break; }
    }
    if (first < 0) {
      first = nbins++;
      resid[first] = capacity;
    }
    bin_of[it[k].idx] = first;
    lane_of[it[k].idx] = capacity - resid[first];
    resid[first] -= s;
  }
  free(resid);
  free(it);
  return nbins;
}

/*
 * Next-Fit: items in path order within each group (groups ascending); one bin
 * is open at a time, and an item that does not fit in it closes it and opens
 * a new one.  A new group always starts a new bin.  Same outputs as
 * or_pack_bfd.
 */
OR_EXPORT int64_t or_pack_nf(int64_t n, const int32_t *size,
                             const int32_t *group, int32_t capacity,
                             int64_t *bin_of, int32_t *lane_of) {
  for (int64_t p = 0; p < n; p++)
    if (size[p] < 1 || size[p] > capacity) return -1;
  int64_t nbins = 0;
  /* groups ascending: visit the distinct group ids in increasing order */
  int32_t g = INT32_MIN;
  for (;;) {
    int found = 0;
    int32_t next = 0;
    for (int64_t p = 0; p < n; p++)
      if (group[p] > g && (!found || group[p] < next)) { next = group[p]; found = 1; }
    if (!found) break;
    g = next;
    int32_t resid = -1; /* no open bin in this group yet */
    for (int64_t p = 0; p < n; p++) {
      if (group[p] != g) continue;
      if (resid < size[p]) {
        nbins++;
        resid = capacity;
      }
      bin_of[p] = nbins - 1;
      lane_of[p] = capacity - resid;
      resid -= size[p];
    }
  }
  return nbins;
}

/*
 * The "none" baseline of Table 5: every path alone in its own bin, bins in
 * the order of (group, path index).  Same outputs as or_pack_bfd.
 */
OR_EXPORT int64_t or_pack_none(int64_t n, const int32_t *size,
                               const int32_t *group, int32_t capacity,
                               int64_t *bin_of, int32_t *lane_of) {
  for (int64_t p = 0; p < n; p++)
    if (size[p] < 1 || size[p] > capacity) return -1;
  int64_t nbins = 0;
  int32_t g = INT32_MIN;
  for (;;) {
    int found = 0;
    int32_t next = 0;
    for (int64_t p = 0; p < n; p++)
      if (group[p] > g && (!found || group[p] < next)) { next = group[p]; found = 1; }
    if (!found) break;
    g = next;
    for (int64_t p = 0; p < n; p++) {
      if (group[p] != g) continue;
      bin_of[p] = nbins++;
      lane_of[p] = 0;
    }
  }
  return nbins;
}
