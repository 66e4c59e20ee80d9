/*
 * np_oracle.c -- TEST INFRASTRUCTURE.  A plain, slow, obviously correct CPU
 * statement of what the NeuroPrefetcher decode hot path computes
 * (arXiv 2608.22643).  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark load this library; the product path never
 * does.  It shares no code with the HIP library or its headers.
 *
 * Floating point: every sum is accumulated in double and rounded once to the
 * output type with round-to-nearest-even.  Conversions between the storage
 * types (IEEE binary16, bfloat16, binary32) and double are written here from
 * the IEEE 754 encodings.
 *
 * Pins (what fixes each function independently of this file) live in the
 * CPU tests: a brute-force sort for selection, an ordered-dict LRU simulator
 * and the set equations for the delta, dense products for the predictor and
 * MLP, a dyadic configuration in which every sum is exact, and numpy's
 * binary16 conversion for the encodings.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_F32 0
#define ORC_F16 1
#define ORC_BF16 2

/* ---------------- IEEE 754 decoding ------------------------------------ */

/* binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits. */
static double orc_from_f16(uint16_t h) {
  int s = (h >> 15) & 1, e = (h >> 10) & 0x1F, f = h & 0x3FF;
  double v;
  if (e == 0)
    v = ldexp((double)f, -24); /* subnormal: f * 2^-14 * 2^-10 */
  else if (e == 31)
    v = f ? NAN : INFINITY;
  else
    v = ldexp((double)(1024 + f), e - 25); /* 1.f * 2^(e-15) */
  return s ? -v : v;
}

/* bfloat16: the upper 16 bits of a binary32 (8 exponent bits, bias 127). */
static double orc_from_bf16(uint16_t b) {
  int s = (b >> 15) & 1, e = (b >> 7) & 0xFF, f = b & 0x7F;
  double v;
  if (e == 0)
    v = ldexp((double)f, -133); /* f * 2^-126 * 2^-7 */
  else if (e == 255)
    v = f ? NAN : INFINITY;
  else
    v = ldexp((double)(128 + f), e - 134); /* 1.f * 2^(e-127) */
  return s ? -v : v;
}

static double orc_from_f32(uint32_t u) {
  int s = (u >> 31) & 1, e = (u >> 23) & 0xFF;
  uint32_t f = u & 0x7FFFFF;
  double v;
  if (e == 0)
    v = ldexp((double)f, -149);
  else if (e == 255)
    v = f ? NAN : INFINITY;
  else
    v = ldexp((double)(0x800000u + f), e - 150);
  return s ? -v : v;
}

static double orc_load(int dtype, const void* p, size_t i) {
  if (dtype == ORC_F32) {
    uint32_t u;
    memcpy(&u, (const char*)p + 4 * i, 4);
    return orc_from_f32(u);
  }
  uint16_t h;
  memcpy(&h, (const char*)p + 2 * i, 2);
  return dtype == ORC_F16 ? orc_from_f16(h) : orc_from_bf16(h);
}

/* ---------------- rounding a double to a narrower format --------------- */

/* Rounds |v| (finite, > 0) to a binary format with `p` significand bits
 * (hidden bit included), minimum normal exponent emin and maximum finite
 * exponent emax, ties to even.  Returns the rounded magnitude as a double
 * (possibly +inf).  Works on the exact binary expansion of v: v = M * 2^E
 * with M the 53-bit integer significand of the double. */
static double orc_round_mag(double a, int p, int emin, int emax) {
  int e2;
  (void)frexp(a, &e2);          /* a in [2^(e2-1), 2^e2) */
  int ex = e2 - 1;              /* a = 1.xxx * 2^ex */
  if (ex < emin) ex = emin;     /* subnormal: fixed quantum */
  int q = ex - (p - 1);         /* quantum of the target grid: 2^q */
  double scaled = ldexp(a, -q); /* exact: power-of-two scaling */
  double lo = floor(scaled);
  double frac = scaled - lo;    /* exact */
  double r = lo;
  if (frac > 0.5 || (frac == 0.5 && fmod(lo, 2.0) != 0.0)) r = lo + 1.0;
  double out = ldexp(r, q);
  double maxfin = ldexp(2.0 - ldexp(1.0, 1 - p), emax);
  if (out > maxfin) return INFINITY;
  return out;
}

static double orc_round_to(int dtype, double v) {
  if (isnan(v) || isinf(v) || v == 0.0) return v;
  double a = fabs(v), r;
  if (dtype == ORC_F32)
    r = orc_round_mag(a, 24, -126, 127);
  else if (dtype == ORC_F16)
    r = orc_round_mag(a, 11, -14, 15);
  else
    r = orc_round_mag(a, 8, -126, 127);
  return v < 0 ? -r : r;
}

/* Bits of an exactly representable value (the result of orc_round_to). */
static uint32_t orc_bits_of(int dtype, double r) {
  int neg = signbit(r) ? 1 : 0;
  double a = fabs(r);
  if (dtype == ORC_F32) {
    uint32_t s = (uint32_t)neg << 31;
    if (isnan(a)) return 0x7FC00000u;
    if (isinf(a)) return s | 0x7F800000u;
    if (a == 0.0) return s;
    int e2;
    (void)frexp(a, &e2);
    int ex = e2 - 1;
    if (ex < -126) return s | (uint32_t)ldexp(a, 149); /* subnormal */
    uint32_t frac = (uint32_t)(ldexp(a, 23 - ex) - 8388608.0);
    return s | ((uint32_t)(ex + 127) << 23) | frac;
  }
  int fbits = dtype == ORC_F16 ? 10 : 7;
  int bias = dtype == ORC_F16 ? 15 : 127;
  int emax_field = dtype == ORC_F16 ? 31 : 255;
  uint32_t s = (uint32_t)neg << 15;
  if (isnan(a)) return dtype == ORC_F16 ? 0x7E00u : 0x7FC0u;
  if (isinf(a)) return s | ((uint32_t)emax_field << fbits);
  if (a == 0.0) return s;
  int e2;
  (void)frexp(a, &e2);
  int ex = e2 - 1;
  if (ex < 1 - bias) /* subnormal: a = f * 2^(1-bias-fbits) */
    return s | (uint32_t)ldexp(a, bias - 1 + fbits);
  uint32_t frac = (uint32_t)(ldexp(a, fbits - ex) - ldexp(1.0, fbits));
  return s | ((uint32_t)(ex + bias) << fbits) | frac;
}

static void orc_store(int dtype, void* p, size_t i, double v) {
  uint32_t b = orc_bits_of(dtype, orc_round_to(dtype, v));
  if (dtype == ORC_F32) {
    memcpy((char*)p + 4 * i, &b, 4);
  } else {
    uint16_t h = (uint16_t)b;
    memcpy((char*)p + 2 * i, &h, 2);
  }
}

void orc_decode(int dtype, const void* in, int64_t n, double* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_load(dtype, in, (size_t)i);
}

void orc_encode(int dtype, const double* in, int64_t n, void* out) {
  for (int64_t i = 0; i < n; ++i) orc_store(dtype, out, (size_t)i, in[i]);
}

/* ---------------- O1: the low-rank activity predictor ------------------ */
/* Sec. 3.1 step 2 and Sec. 3.3: one predictor pass after layer 0 scores the
 * MLP neurons of all downstream layers.  Low-rank form per layer l:
 * z_l = A_l h (length r, left unrounded), scores_l = fp32(B_l z_l). */
int orc_predict(int L, int d, int F, int r, int wdtype, int adtype,
                const void* h, const void* A, const void* B, float* scores) {
  double* hv = (double*)malloc(sizeof(double) * (size_t)d);
  double* z = (double*)malloc(sizeof(double) * (size_t)r);
  if (!hv || !z) { free(hv); free(z); return -1; }
  for (int c = 0; c < d; ++c) hv[c] = orc_load(adtype, h, (size_t)c);
  for (int l = 0; l < L; ++l) {
    for (int j = 0; j < r; ++j) {
      double acc = 0.0;
      size_t row = ((size_t)l * r + j) * d;
      for (int c = 0; c < d; ++c) acc += orc_load(wdtype, A, row + c) * hv[c];
      z[j] = acc;
    }
    for (int n = 0; n < F; ++n) {
      double acc = 0.0;
      size_t row = ((size_t)l * F + n) * r;
      for (int j = 0; j < r; ++j) acc += orc_load(wdtype, B, row + j) * z[j];
      double rounded = orc_round_to(ORC_F32, acc);
      scores[(size_t)l * F + n] = (float)rounded; /* exact: already on grid */
    }
  }
  free(hv);
  free(z);
  return 0;
}

/* ---------------- O2: top-k into fixed-size active sets ---------------- */
/* Sec. 3.4: every active set has the same size.  The active set is the k
 * neurons with the largest score; a tie at the k-th score goes to the
 * smaller id; -0 and +0 are equal; a NaN score is an error. */
/* The comparator's scores: qsort passes no context, so the array is handed
 * over in a thread-local pointer (calls from several threads stay apart). */
static _Thread_local const float* g_sort_scores;

static int by_score_desc_id_asc(const void* pa, const void* pb) {
  int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
  double sa = g_sort_scores[a], sb = g_sort_scores[b];
  if (sa > sb) return -1;
  if (sa < sb) return 1;
  return a < b ? -1 : (a > b ? 1 : 0);
}

static int by_int_asc(const void* pa, const void* pb) {
  int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
  return a < b ? -1 : (a > b ? 1 : 0);
}

int orc_select(int L, int F, int k, const float* scores, uint32_t* mask,
               int32_t* active_ids) {
  int words = (F + 31) / 32;
  int32_t* order = (int32_t*)malloc(sizeof(int32_t) * (size_t)F);
  if (!order) return -1;
  for (int l = 0; l < L; ++l) {
    const float* s = scores + (size_t)l * F;
    for (int n = 0; n < F; ++n) {
      if (isnan(s[n])) { free(order); return 1; }
      order[n] = n;
    }
    g_sort_scores = s;
    qsort(order, (size_t)F, sizeof(int32_t), by_score_desc_id_asc);
    int32_t* ids = active_ids + (size_t)l * k;
    memcpy(ids, order, sizeof(int32_t) * (size_t)k);
    qsort(ids, (size_t)k, sizeof(int32_t), by_int_asc);
    uint32_t* m = mask + (size_t)l * words;
    memset(m, 0, sizeof(uint32_t) * (size_t)words);
    for (int j = 0; j < k; ++j) m[ids[j] / 32] |= 1u << (ids[j] % 32);
  }
  free(order);
  return 0;
}

/* ---------------- O3: delta against the resident set ------------------- */
/* Sec. 3.4, eqs. (2)-(3) and the slot-map paragraph, generalised to a
 * resident buffer of C >= k slots:
 *   hits H = {n in A : P[n] >= 0}, incoming I = A \ H (ascending);
 *   free slots Fr = {s : Q[s] = -1} (ascending);
 *   if |I| <= |Fr| the pool is the first |I| free slots and nothing leaves;
 *   otherwise the m = |I| - |Fr| victims V are the resident neurons outside A
 *   with the smallest (U[n], n), and the pool is Fr together with the
 *   victims' slots, ascending;
 *   victims release their slots (P[n] = -1, Q[s] = -1), I[j] takes pool[j],
 *   U[n] = t for every n in A.
 * P = slot_of [L][F], Q = neuron_of [L][C], U = last_used [L][F].
 * Outputs are [L][k] lists (first counts entries defined) and counts [L][4].
 * Returns 0, or 2 if a precondition fails (A not strictly ascending or out
 * of range, P and Q not mutual inverses, k > C). */
static _Thread_local const int32_t* g_sort_lastused;  /* as g_sort_scores */

static int by_lastused_then_id(const void* pa, const void* pb) {
  int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
  int32_t ua = g_sort_lastused[a], ub = g_sort_lastused[b];
  if (ua != ub) return ua < ub ? -1 : 1;
  return a < b ? -1 : (a > b ? 1 : 0);
}

/* active_counts: NULL for k active neurons per layer, else n_l <= k of them
 * (active_ids[l][0..n_l) ascending) -- the variable-size sets of the
 * centroid predictor (Sec. 3.4: the intersection of two masks). */
static int orc_delta_impl(int L, int F, int C, int k, int32_t t, const int32_t* active_ids,
                          const int32_t* active_counts, int32_t* slot_of, int32_t* neuron_of,
                          int32_t* last_used, int32_t* in_ids, int32_t* in_slots,
                          int32_t* ev_ids, int32_t* ev_slots, int32_t* hit_ids,
                          int32_t* active_slots, int32_t* counts) {
  if (k > C) return 2;
  char* in_a = (char*)malloc((size_t)F);
  int32_t* fr = (int32_t*)malloc(sizeof(int32_t) * (size_t)C);
  int32_t* cand = (int32_t*)malloc(sizeof(int32_t) * (size_t)F);
  int32_t* pool = (int32_t*)malloc(sizeof(int32_t) * (size_t)(C + k));
  if (!in_a || !fr || !cand || !pool) {
    free(in_a); free(fr); free(cand); free(pool);
    return -1;
  }
  int rc = 0;
  for (int l = 0; l < L && rc == 0; ++l) {
    const int32_t* A = active_ids + (size_t)l * k;
    int32_t* P = slot_of + (size_t)l * F;
    int32_t* Q = neuron_of + (size_t)l * C;
    int32_t* U = last_used + (size_t)l * F;
    int32_t* I = in_ids + (size_t)l * k;
    int32_t* IS = in_slots + (size_t)l * k;
    int32_t* V = ev_ids + (size_t)l * k;
    int32_t* VS = ev_slots + (size_t)l * k;
    int32_t* H = hit_ids + (size_t)l * k;
    int32_t* AS = active_slots + (size_t)l * k;
    const int na = active_counts ? active_counts[l] : k;

    /* preconditions */
    if (na < 0 || na > k) rc = 2;
    for (int j = 0; j < na && rc == 0; ++j) {
      if (A[j] < 0 || A[j] >= F || (j > 0 && A[j] <= A[j - 1])) rc = 2;
    }
    for (int n = 0; n < F && rc == 0; ++n)
      if (P[n] >= 0 && (P[n] >= C || Q[P[n]] != n)) rc = 2;
    for (int s = 0; s < C && rc == 0; ++s)
      if (Q[s] >= 0 && (Q[s] >= F || P[Q[s]] != s)) rc = 2;
    if (rc) break;

    memset(in_a, 0, (size_t)F);
    for (int j = 0; j < na; ++j) in_a[A[j]] = 1;

    int nh = 0, ni = 0;
    for (int j = 0; j < na; ++j) {
      if (P[A[j]] >= 0) H[nh++] = A[j];
      else I[ni++] = A[j];
    }
    int nfree = 0;
    for (int s = 0; s < C; ++s)
      if (Q[s] == -1) fr[nfree++] = s;

    int nv = 0, npool = 0;
    if (ni <= nfree) {
      for (int j = 0; j < ni; ++j) pool[npool++] = fr[j];
    } else {
      int m = ni - nfree, nc = 0;
      for (int n = 0; n < F; ++n)
        if (P[n] >= 0 && !in_a[n]) cand[nc++] = n;
      if (nc < m) { rc = 2; break; }
      g_sort_lastused = U;
      qsort(cand, (size_t)nc, sizeof(int32_t), by_lastused_then_id);
      for (int j = 0; j < m; ++j) V[nv++] = cand[j];
      qsort(V, (size_t)nv, sizeof(int32_t), by_int_asc);
      for (int j = 0; j < nfree; ++j) pool[npool++] = fr[j];
      for (int j = 0; j < nv; ++j) pool[npool++] = P[V[j]];
      qsort(pool, (size_t)npool, sizeof(int32_t), by_int_asc);
    }
    for (int j = 0; j < nv; ++j) VS[j] = P[V[j]];
    for (int j = 0; j < nv; ++j) {
      Q[P[V[j]]] = -1;
      P[V[j]] = -1;
    }
    for (int j = 0; j < ni; ++j) {
      IS[j] = pool[j];
      P[I[j]] = pool[j];
      Q[pool[j]] = I[j];
    }
    for (int j = 0; j < na; ++j) U[A[j]] = t;
    for (int j = 0; j < na; ++j) AS[j] = P[A[j]];
    int32_t* cnt = counts + (size_t)l * 4;
    cnt[0] = ni;
    cnt[1] = nh;
    cnt[2] = nv;
    cnt[3] = ni - nv;
  }
  free(in_a);
  free(fr);
  free(cand);
  free(pool);
  return rc;
}

int orc_delta(int L, int F, int C, int k, int32_t t, const int32_t* active_ids,
              int32_t* slot_of, int32_t* neuron_of, int32_t* last_used,
              int32_t* in_ids, int32_t* in_slots, int32_t* ev_ids,
              int32_t* ev_slots, int32_t* hit_ids, int32_t* active_slots,
              int32_t* counts) {
  return orc_delta_impl(L, F, C, k, t, active_ids, NULL, slot_of, neuron_of, last_used, in_ids,
                        in_slots, ev_ids, ev_slots, hit_ids, active_slots, counts);
}

int orc_delta_n(int L, int F, int C, int k, int32_t t, const int32_t* active_ids,
                const int32_t* active_counts, int32_t* slot_of, int32_t* neuron_of,
                int32_t* last_used, int32_t* in_ids, int32_t* in_slots, int32_t* ev_ids,
                int32_t* ev_slots, int32_t* hit_ids, int32_t* active_slots, int32_t* counts) {
  return orc_delta_impl(L, F, C, k, t, active_ids, active_counts, slot_of, neuron_of, last_used,
                        in_ids, in_slots, ev_ids, ev_slots, hit_ids, active_slots, counts);
}

/* ---------------- O4: staging -------------------------------------------- */
/* Sec. 3.5: each incoming neuron's record (gate, up and down^T rows, 3d
 * elements) lands in the slot the delta assigned to it.  A byte copy. */
void orc_stage(int L, int F, int C, int k, int d, int wdtype,
               const int32_t* counts, const int32_t* in_ids,
               const int32_t* in_slots, const void* storage, void* resident) {
  size_t rec = (size_t)3 * d * (wdtype == ORC_F32 ? 4 : 2);
  for (int l = 0; l < L; ++l) {
    int n_in = counts[(size_t)l * 4];
    for (int j = 0; j < n_in; ++j) {
      size_t src = ((size_t)l * F + in_ids[(size_t)l * k + j]) * rec;
      size_t dst = ((size_t)l * C + in_slots[(size_t)l * k + j]) * rec;
      memcpy((char*)resident + dst, (const char*)storage + src, rec);
    }
  }
}

/* ---------------- gated activations and eq. 1 ---------------------------- */
/* The two gated forms of an MLP neuron with gate sum g and up sum u:
 *   ReLU-gated (the synthetic models):  a = max(g, 0) * u;
 *   SwiGLU (the paper's evaluated models, Sec. 4):  a = SiLU(g) * u with
 *   SiLU(g) = g * sigmoid(g) = g / (1 + e^-g)  (exp from the C library).
 * Eq. 1 (Sec. 3.2): a magnitude below the layer's threshold T is set to zero;
 * T = 0 leaves every value as it is. */
#define ORC_ACT_RELU 0
#define ORC_ACT_SWIGLU 1

static double orc_act(int act, double g, double u) {
  if (act == ORC_ACT_SWIGLU) return g / (1.0 + exp(-g)) * u;
  return (g > 0.0 ? g : 0.0) * u;
}

static double orc_eq1(double a, double thr) { return fabs(a) < thr ? 0.0 : a; }

/* ---------------- O5: sparse MLP over the active rows ------------------ */
/* Sec. 3.4 (row i of gate, up and down^T for each active neuron; row order
 * irrelevant) and Sec. 3.3 (the down projection's output stays dense).
 * Computed from the storage tier, indexed by neuron id -- the definition, not
 * the resident buffer.  y = sum over n in ids of eq1(act(G[n].x, U[n].x)) *
 * D[n] with the activation `act` and threshold `thr` above; y is rounded once
 * to adtype; y64 (optional) receives the unrounded sums. */
int orc_sparse_mlp(int F, int d, int wdtype, int adtype, int act, double thr, int layer,
                   const void* x, const void* storage, const int32_t* ids,
                   int n_ids, void* y, double* y64) {
  double* xv = (double*)malloc(sizeof(double) * (size_t)d);
  double* acc = (double*)calloc((size_t)d, sizeof(double));
  if (!xv || !acc) { free(xv); free(acc); return -1; }
  for (int c = 0; c < d; ++c) xv[c] = orc_load(adtype, x, (size_t)c);
  for (int j = 0; j < n_ids; ++j) {
    int n = ids[j];
    if (n < 0 || n >= F) { free(xv); free(acc); return 2; }
    size_t base = ((size_t)layer * F + n) * 3 * (size_t)d;
    double g = 0.0, u = 0.0;
    for (int c = 0; c < d; ++c) {
      g += orc_load(wdtype, storage, base + c) * xv[c];
      u += orc_load(wdtype, storage, base + d + c) * xv[c];
    }
    double a = orc_eq1(orc_act(act, g, u), thr);
    for (int c = 0; c < d; ++c)
      acc[c] += a * orc_load(wdtype, storage, base + 2 * (size_t)d + c);
  }
  for (int c = 0; c < d; ++c) {
    if (y) orc_store(adtype, y, (size_t)c, acc[c]);
    if (y64) y64[c] = acc[c];
  }
  free(xv);
  free(acc);
  return 0;
}

/* ---------------- O6: dense MLP, matrix form ----------------------------- */
/* The same MLP over all F neurons, written as whole-matrix products:
 * gvec = G x, uvec = U x, avec = eq1(act(gvec, uvec)), y = D^T avec.  Pins
 * O5 (all neurons active must give the dense result) and is the dense
 * layer of the dense prefix (Sec. 3.1). */
int orc_dense_mlp(int F, int d, int wdtype, int adtype, int act, double thr, int layer,
                  const void* x, const void* storage, void* y, double* y64) {
  double* xv = (double*)malloc(sizeof(double) * (size_t)d);
  double* gv = (double*)malloc(sizeof(double) * (size_t)F);
  double* uv = (double*)malloc(sizeof(double) * (size_t)F);
  double* yv = (double*)malloc(sizeof(double) * (size_t)d);
  if (!xv || !gv || !uv || !yv) {
    free(xv); free(gv); free(uv); free(yv);
    return -1;
  }
  size_t lbase = (size_t)layer * F * 3 * (size_t)d;
  for (int c = 0; c < d; ++c) xv[c] = orc_load(adtype, x, (size_t)c);
  /* gvec and uvec: row n of G (U) is the first (second) d elements of record n */
  for (int n = 0; n < F; ++n) {
    double sg = 0.0, su = 0.0;
    for (int c = 0; c < d; ++c) {
      sg += orc_load(wdtype, storage, lbase + (size_t)n * 3 * d + c) * xv[c];
      su += orc_load(wdtype, storage, lbase + (size_t)n * 3 * d + d + c) * xv[c];
    }
    gv[n] = sg;
    uv[n] = su;
  }
  /* y[c] = sum_n D^T[n][c] * act[n], column by column */
  for (int c = 0; c < d; ++c) {
    double s = 0.0;
    for (int n = 0; n < F; ++n) {
      double an = orc_eq1(orc_act(act, gv[n], uv[n]), thr);
      s += orc_load(wdtype, storage, lbase + (size_t)n * 3 * d + 2 * (size_t)d + c) * an;
    }
    yv[c] = s;
  }
  for (int c = 0; c < d; ++c) {
    if (y) orc_store(adtype, y, (size_t)c, yv[c]);
    if (y64) y64[c] = yv[c];
  }
  free(xv); free(gv); free(uv); free(yv);
  return 0;
}

/* ---------------- O7: centroid-ID heads ---------------------------------- */
/* Sec. 3.3 (architecture, third stage): two groups of L' linear heads map the
 * predictor's feature vector to gate and up logits over K centroids.  Head h
 * (0..H-1; gate heads of layers 0..L'-1, then up heads) is a K x D matrix:
 * logits[h][c] = heads[h][c] . feat, summed in double, rounded to binary32. */
int orc_centroid_logits(int H, int K, int D, int wdtype, int adtype, const void* heads,
                        const void* feat, float* logits) {
  double* f = (double*)malloc(sizeof(double) * (size_t)D);
  if (!f) return -1;
  for (int i = 0; i < D; ++i) f[i] = orc_load(adtype, feat, (size_t)i);
  for (int64_t row = 0; row < (int64_t)H * K; ++row) {
    double acc = 0.0;
    for (int i = 0; i < D; ++i) acc += orc_load(wdtype, heads, (size_t)row * D + i) * f[i];
    logits[row] = (float)orc_round_to(ORC_F32, acc);
  }
  free(f);
  return 0;
}

/* ---------------- O8: centroid choice and the intersected active set ----- */
/* Sec. 3.3: each head selects its highest-scoring centroid (a tie goes to the
 * smaller index).  Sec. 3.4: the active set of layer l is the intersection of
 * the chosen gate and up centroid masks.  bank [2][L'][K][W] holds the masks
 * (W = ceil(F/32) words, bit n%32 of word n/32), gate masks first.  Outputs:
 * cids [2][L'] (gate ids, then up ids), mask [L'][W] (the intersection),
 * active_ids [L'][k] ascending, counts [L'].  The list of a layer holds at
 * most k ids (its buffer capacity): a larger intersection keeps its k
 * smallest ids, its mask keeps every member, and the function returns 3.
 * A NaN logit returns 1 (nothing else is checked for it). */
int orc_centroid_active(int L, int F, int K, int k, const float* logits, const uint32_t* bank,
                        int32_t* cids, uint32_t* mask, int32_t* active_ids, int32_t* counts) {
  const int W = (F + 31) / 32;
  int rc = 0;
  for (int h = 0; h < 2 * L; ++h) {
    const float* lg = logits + (size_t)h * K;
    int best = 0;
    for (int c = 0; c < K; ++c) {
      if (isnan(lg[c])) return 1;
      if (lg[c] > lg[best]) best = c;  /* strict: the first maximum wins */
    }
    cids[h] = best;
  }
  for (int l = 0; l < L; ++l) {
    const uint32_t* g = bank + ((size_t)l * K + cids[l]) * W;
    const uint32_t* u = bank + (((size_t)L + l) * K + cids[L + l]) * W;
    int n = 0;
    for (int w = 0; w < W; ++w) {
      uint32_t m = g[w] & u[w];
      if (w == W - 1 && (F & 31)) m &= (1u << (F & 31)) - 1u;
      mask[(size_t)l * W + w] = m;
      for (int b = 0; b < 32; ++b) {
        if (!((m >> b) & 1u)) continue;
        if (n < k) active_ids[(size_t)l * k + n] = 32 * w + b;
        ++n;
      }
    }
    if (n > k) {
      rc = 3;
      n = k;
    }
    counts[l] = n;
  }
  return rc;
}

/* ---------------- O9: activations of a batch of tokens -------------------- */
/* Sec. 3.2: the activations A_i = f_l(x_i) of layer l over tokens x_i, the
 * input of the percentile calibration.  weights is one layer's [F][3d]
 * records, x is [n][d]; acts[i][f] = act(G[f].x_i, U[f].x_i) in double,
 * unrounded. */
int orc_act_batch(int F, int d, int wdtype, int adtype, int act, const void* weights,
                  const void* x, int n, double* acts) {
  double* xv = (double*)malloc(sizeof(double) * (size_t)d);
  if (!xv) return -1;
  for (int i = 0; i < n; ++i) {
    for (int c = 0; c < d; ++c) xv[c] = orc_load(adtype, x, (size_t)i * d + c);
    for (int f = 0; f < F; ++f) {
      size_t base = (size_t)f * 3 * d;
      double g = 0.0, u = 0.0;
      for (int c = 0; c < d; ++c) {
        g += orc_load(wdtype, weights, base + c) * xv[c];
        u += orc_load(wdtype, weights, base + d + c) * xv[c];
      }
      acts[(size_t)i * F + f] = orc_act(act, g, u);
    }
  }
  free(xv);
  return 0;
}

/* ---------------- O10: the alpha-th percentile of the magnitudes ---------- */
/* Sec. 3.2: T(l, alpha) is the alpha-th percentile of |A| over the
 * calibration activations of layer l.  Reading: the nearest-rank percentile,
 * the m-th smallest magnitude with m = ceil(alpha * n / 100) evaluated in
 * double and clamped to [1, n]; it is a value of the set itself, so eq. 1
 * then zeroes fewer than m of the n values.  values: [rows][n] binary32, one
 * row per layer; out: [rows].  alpha outside [0, 100] or n < 1 returns 2, a
 * NaN value returns 1. */
static int by_float_asc(const void* pa, const void* pb) {
  float a = *(const float*)pa, b = *(const float*)pb;
  return a < b ? -1 : (a > b ? 1 : 0);
}

int64_t orc_percentile_rank(int64_t n, double alpha) {
  double m = ceil(alpha * (double)n / 100.0);
  if (m < 1.0) m = 1.0;
  if (m > (double)n) m = (double)n;
  return (int64_t)m;
}

int orc_percentile(const float* values, int rows, int64_t n, double alpha, float* out) {
  if (n < 1 || !(alpha >= 0.0 && alpha <= 100.0)) return 2;
  float* mag = (float*)malloc(sizeof(float) * (size_t)n);
  if (!mag) return -1;
  int64_t m = orc_percentile_rank(n, alpha);
  for (int r = 0; r < rows; ++r) {
    for (int64_t i = 0; i < n; ++i) {
      float v = values[(size_t)r * n + i];
      if (isnan(v)) { free(mag); return 1; }
      mag[i] = fabsf(v);
    }
    qsort(mag, (size_t)n, sizeof(float), by_float_asc);
    out[r] = mag[m - 1];
  }
  free(mag);
  return 0;
}

/* ---------------- O11: the thresholded active set ------------------------ */
/* Eq. 1 as a mask: neuron f of row r is active when |acts[r][f]| >= thr[r]
 * (what eq. 1 keeps), in the layout of the selection: mask [rows][W] (bit
 * f%32 of word f/32), active_ids [rows][k] ascending, counts [rows].  A row
 * with more than k active neurons keeps its k smallest ids in the list and
 * every member in the mask, and the function returns 3; a NaN returns 1. */
int orc_threshold_active(int rows, int F, int k, const float* acts, const float* thr,
                         uint32_t* mask, int32_t* active_ids, int32_t* counts) {
  const int W = (F + 31) / 32;
  int rc = 0;
  for (int r = 0; r < rows; ++r) {
    int n = 0;
    for (int w = 0; w < W; ++w) mask[(size_t)r * W + w] = 0u;
    for (int f = 0; f < F; ++f) {
      float v = acts[(size_t)r * F + f];
      if (isnan(v)) return 1;
      if (fabsf(v) >= thr[r]) {
        mask[(size_t)r * W + f / 32] |= 1u << (f % 32);
        if (n < k) active_ids[(size_t)r * k + n] = f;
        ++n;
      }
    }
    if (n > k) {
      rc = 3;
      n = k;
    }
    counts[r] = n;
  }
  return rc;
}
