/*
 * Reference oracle for the LRAM lattice lookup -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow CPU code that computes the truncated lattice lookup straight
 * from its definition.  It is used by the test-suite, by the smoke check and
 * by the CPU-baseline leg of the benchmark; the product path never links,
 * loads or calls it.  It shares no code, header or table with the GPU
 * library: in particular it knows nothing of the symmetry reduction, the
 * fundamental region or the 232-point candidate table, it simply enumerates
 * every lattice point near the query.
 *
 * Definitions followed (Goucher & Troll, "Differentiable Random Access Memory
 * using Lattices"):
 *   - Sec. 2.2 (Mathematical Formulation): torus T_K = R^8 / L_K, memory
 *     locations M = Lambda / L_K, lookup phi(q) = sum_k f(d(q,k)) v_k.
 *   - Sec. 2.4 (Choice of Lattice): Lambda = { x in (2Z)^8 u (2Z+1)^8 :
 *     sum x_i = 0 mod 4 }, i.e. E8 at twice the unimodular scale.
 *   - Sec. 2.5 (Choice of Kernel): f(r) = max(0, 1 - r^2/8)^4, support r^2 < 8.
 *   - Sec. 2.6 (Implementation): all lattice points at distance < sqrt(8),
 *     truncated to the closest 32.
 *
 * Readings this build takes where the paper is silent (each is listed with
 * its reason in the design notes):
 *   - User scale: the caller passes q with coordinates in [0, K_i) on a
 *     unimodular-E8 torus of side K_i; the Lambda-scale point is
 *     x_i = fmodf(2 q_i, 2 K_i) (exact, sign kept).  N = prod K_i locations,
 *     every K_i even and >= 2.
 *   - Lift semantics: the sum runs over lattice points k of Lambda in R^8
 *     (not over torus classes); each k is mapped to its location.  For
 *     every K_i >= 4 this equals the quotient-metric sum of Sec. 2.2.
 *   - Distance recipe (decides which 32 points are kept, so both the oracle
 *     and the GPU take it in the same fp32 arithmetic):
 *       e_i = fl32(x_i - (float)k_i);  s = e_0*e_0;  s = fl32(s + fl32(e_i*e_i))
 *       for i = 1..7 in coordinate order; round-to-nearest-even, no FMA.
 *     A point is in the support iff s < 8 (open ball).
 *   - Order: ascending (bits(s), slot, k lexicographic).  Keep the first
 *     min(32, count); pad with slot -1, weight 0.
 *   - Location bijection: eps = k_0 mod 2; Y_i = ((k_i - eps)/2) mod K_i
 *     (floor mod); slot = eps*N/2 + ((..(Y_0 K_1 + Y_1) K_2 + ..) K_6 + Y_6)
 *     * (K_7/2) + floor(Y_7/2).
 *   - A non-finite query coordinate gives an empty neighbour list.
 *
 * Weights are reported twice: the fp64 value f(r) with r^2 taken in fp64
 * from the exact differences (the "truth"), and the fp32 value of the
 * recipe u = fl(1 - s*0.125f), w = fl(fl(u*u)*fl(u*u)) for bit-level checks.
 *
 * Build: gcc -O2 -fPIC -shared -fopenmp -ffp-contract=off (the contract flag
 * matters: the fp32 recipe must not be fused into FMAs).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_NB 32
#define ORACLE_MAXPTS 512

typedef struct {
  float d;       /* recipe distance^2, fp32 */
  int32_t slot;  /* location index */
  int32_t k[8];  /* the lattice point (a lift in R^8), Lambda scale */
  double d64;    /* distance^2 in fp64 */
} rec_t;

static int cmp_rec(const void* a, const void* b) {
  const rec_t* x = (const rec_t*)a;
  const rec_t* y = (const rec_t*)b;
  uint32_t bx, by;
  memcpy(&bx, &x->d, 4);
  memcpy(&by, &y->d, 4);
  if (bx != by) return bx < by ? -1 : 1;
  if (x->slot != y->slot) return x->slot < y->slot ? -1 : 1;
  for (int i = 0; i < 8; i++)
    if (x->k[i] != y->k[i]) return x->k[i] < y->k[i] ? -1 : 1;
  return 0;
}

/* The fp32 distance recipe, coordinates in their original order. */
static float recipe_d2(const float x[8], const int32_t k[8]) {
  float s = 0.0f;
  for (int i = 0; i < 8; i++) {
    float e = x[i] - (float)k[i];
    float sq = e * e;
    if (i == 0)
      s = sq;
    else
      s = s + sq;
  }
  return s;
}

static int64_t floor_mod(int64_t a, int64_t m) {
  int64_t r = a % m;
  return r < 0 ? r + m : r;
}

/* Location of lattice point k on the torus with periods 2*K_i (Lambda scale). */
static int32_t location_of(const int32_t k[8], const int32_t K[8], int64_t N) {
  int64_t eps = floor_mod(k[0], 2);
  int64_t Y[8];
  for (int i = 0; i < 8; i++) Y[i] = floor_mod((k[i] - eps) / 2, K[i]);
  int64_t idx = Y[0];
  for (int i = 1; i < 7; i++) idx = idx * K[i] + Y[i];
  idx = idx * (K[7] / 2) + Y[7] / 2;
  return (int32_t)(eps * (N / 2) + idx);
}

typedef struct {
  const float* x;
  const int32_t* K;
  int64_t N;
  rec_t* out;
  int n;
  int overflow;
} enum_ctx;

/* Depth-first enumeration of one coset of Lambda: every coordinate is
 * k_i = 2t + eps with |x_i - k_i| < sqrt(8) (plus slack), pruned when the fp64
 * partial sum of squares already exceeds 8 (plus slack).  The slack is far
 * larger than any fp32 rounding in the recipe, so no point with recipe
 * distance < 8 is pruned; the recipe test at the leaf decides membership. */
static void enum_coset(enum_ctx* c, int i, int eps, int32_t* k, double partial, int64_t sum) {
  const double R = 2.8284271247461903 + 1e-3;
  const double LIM = 8.0 + 1e-3;
  if (i == 8) {
    if (floor_mod(sum, 4) != 0) return;
    float d = recipe_d2(c->x, k);
    if (!(d < 8.0f)) return;
    if (c->n >= ORACLE_MAXPTS) {
      c->overflow = 1;
      return;
    }
    rec_t* r = &c->out[c->n++];
    r->d = d;
    memcpy(r->k, k, sizeof(int32_t) * 8);
    r->slot = location_of(k, c->K, c->N);
    double d64 = 0.0;
    for (int j = 0; j < 8; j++) {
      double e = (double)c->x[j] - (double)k[j];
      d64 += e * e;
    }
    r->d64 = d64;
    return;
  }
  double xi = (double)c->x[i];
  int64_t t0 = (int64_t)ceil((xi - R - eps) / 2.0);
  int64_t t1 = (int64_t)floor((xi + R - eps) / 2.0);
  for (int64_t t = t0; t <= t1; t++) {
    int64_t ki = 2 * t + eps;
    double e = xi - (double)ki;
    double p = partial + e * e;
    if (p >= LIM) continue;
    k[i] = (int32_t)ki;
    enum_coset(c, i + 1, eps, k, p, sum + ki);
  }
}

static double kernel64(double d2) {
  double u = 1.0 - d2 / 8.0;
  if (u <= 0.0) return 0.0;
  double u2 = u * u;
  return u2 * u2;
}

/*
 * For each of L queries q[L][8] on the torus K[8]:
 *   x      [L][8]   fp32  Lambda-scale wrapped query (output)
 *   count  [L]      int32 size of the full (untruncated) support, 0 if q is not finite
 *   slot   [L][32]  int32 locations of the closest min(32,count) points, -1 padded
 *   d2     [L][32]  fp32  recipe distance^2 (padding: +inf)
 *   d64    [L][32]  fp64  distance^2 in fp64 (padding: 0)
 *   w64    [L][32]  fp64  kernel weight from d64 (padding: 0)
 *   w32    [L][32]  fp32  recipe weight from d2 (padding: 0)
 *   lift   [L][32][8] int32 the lattice points themselves (padding: 0)
 *   wsum   [L]      fp64  total kernel weight over the full support
 * Returns 0, or -1 if some query had more than ORACLE_MAXPTS support points
 * (impossible for E8: at most 241 even on the closed ball).
 * lram_oracle_neighbors_k writes `width` entries per lookup instead of 32:
 * the closest min(width, count) points in the same order (width >= 241 keeps
 * the whole support, i.e. the untruncated sum of Sec. 2.2 / 2.5).
 */
int lram_oracle_neighbors_k(const float* q, int64_t L, const int32_t* K, int32_t width, float* x_out,
                            int32_t* count, int32_t* slot, float* d2, double* d64,
                            double* w64, float* w32, int32_t* lift, double* wsum) {
  int64_t N = 1;
  for (int i = 0; i < 8; i++) N *= K[i];
  int bad = 0;
#pragma omp parallel for schedule(dynamic, 64) reduction(| : bad)
  for (int64_t l = 0; l < L; l++) {
    rec_t recs[ORACLE_MAXPTS];
    float x[8];
    int finite = 1;
    for (int i = 0; i < 8; i++) {
      float qi = q[l * 8 + i];
      x[i] = fmodf(2.0f * qi, 2.0f * (float)K[i]);
      if (!isfinite(x[i])) finite = 0;
      x_out[l * 8 + i] = x[i];
    }
    enum_ctx c = {x, K, N, recs, 0, 0};
    if (finite) {
      int32_t k[8];
      enum_coset(&c, 0, 0, k, 0.0, 0);
      enum_coset(&c, 0, 1, k, 0.0, 0);
      if (c.overflow) bad = 1;
      qsort(recs, (size_t)c.n, sizeof(rec_t), cmp_rec);
    }
    count[l] = c.n;
    double total = 0.0;
    for (int j = 0; j < c.n; j++) total += kernel64(recs[j].d64);
    wsum[l] = total;
    for (int j = 0; j < width; j++) {
      int64_t o = l * width + j;
      if (j < c.n) {
        const rec_t* r = &recs[j];
        slot[o] = r->slot;
        d2[o] = r->d;
        d64[o] = r->d64;
        w64[o] = kernel64(r->d64);
        float u = 1.0f - r->d * 0.125f;
        float u2 = u * u;
        w32[o] = u2 * u2;
        memcpy(&lift[o * 8], r->k, sizeof(int32_t) * 8);
      } else {
        slot[o] = -1;
        d2[o] = INFINITY;
        d64[o] = 0.0;
        w64[o] = 0.0;
        w32[o] = 0.0f;
        memset(&lift[o * 8], 0, sizeof(int32_t) * 8);
      }
    }
  }
  return bad ? -1 : 0;
}

/* The closest-32 lists (Sec. 2.6). */
int lram_oracle_neighbors(const float* q, int64_t L, const int32_t* K, float* x_out,
                          int32_t* count, int32_t* slot, float* d2, double* d64,
                          double* w64, float* w32, int32_t* lift, double* wsum) {
  return lram_oracle_neighbors_k(q, L, K, ORACLE_NB, x_out, count, slot, d2, d64, w64, w32, lift, wsum);
}

/* Location of explicit lattice points (for tests of the bijection). */
void lram_oracle_locations(const int32_t* k, int64_t n, const int32_t* K, int32_t* out) {
  int64_t N = 1;
  for (int i = 0; i < 8; i++) N *= K[i];
  for (int64_t j = 0; j < n; j++) out[j] = location_of(&k[j * 8], K, N);
}

/* The fp32 recipe distance for explicit (x, k) pairs. */
void lram_oracle_recipe_d2(const float* x, const int32_t* k, int64_t n, float* out) {
  for (int64_t j = 0; j < n; j++) out[j] = recipe_d2(&x[j * 8], &k[j * 8]);
}
