/*
 * npgen.c -- seeded synthetic inputs for the NeuroPrefetcher decode path.
 *
 * This file generates inputs only: MLP neuron records, predictor factors,
 * the hidden-state sequence, and the centroid predictor's feature sequence,
 * head matrices and centroid mask bank.  It holds none of the method's arithmetic; both
 * the HIP path and the CPU oracle consume what it writes.
 *
 * Random numbers come from a counter-based generator: value i of the stream
 * (seed, tensor, layer) is the i-th output of SplitMix64 (Steele, Lea and
 * Flood, "Fast splittable pseudorandom number generators", OOPSLA 2014)
 * started from a state derived from (seed, tensor, layer).  Any element can
 * therefore be generated independently, in any order and on any thread.
 * Normal variates use the Box-Muller transform on two consecutive draws
 * (in single precision).
 *
 * Floating-point encodings (fp16 = IEEE binary16, bf16 = the top half of
 * binary32) round to nearest, ties to even, from a double.
 */
#define _GNU_SOURCE /* sincos */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <string.h>

#define NPG_F32 0
#define NPG_F16 1
#define NPG_BF16 2

static const uint64_t GOLDEN = 0x9E3779B97F4A7C15ULL;

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

uint64_t npg_stream(uint64_t seed, uint32_t tensor, uint32_t layer) {
  uint64_t s = mix64(seed + GOLDEN * ((uint64_t)tensor + 1));
  return mix64(s + GOLDEN * ((uint64_t)layer + 1));
}

/* i-th SplitMix64 output of a generator whose state starts at `stream`. */
uint64_t npg_draw(uint64_t stream, uint64_t i) {
  return mix64(stream + GOLDEN * (i + 1));
}

/* Uniform on the open interval (0, 1): 53 random bits, centred in their cell. */
static inline double unit_open(uint64_t x) {
  return ((double)(x >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}

/* Box-Muller: elements 2m and 2m+1 of a stream are the cosine and sine
 * outputs of the uniform pair (draw 2m, draw 2m+1). */
static inline void normal_pair(uint64_t stream, uint64_t m, double* z0, double* z1) {
  /* single-precision transcendental functions: the variates are stored in
   * 16-bit or 32-bit formats, far coarser than float's rounding error */
  const float u1 = (float)unit_open(npg_draw(stream, 2 * m));
  const float u2 = (float)unit_open(npg_draw(stream, 2 * m + 1));
  const float r = sqrtf(-2.0f * logf(u1));
  float sn, cs;
  sincosf(6.28318530717958647692f * u2, &sn, &cs);
  *z0 = (double)(r * cs);
  *z1 = (double)(r * sn);
}

double npg_normal(uint64_t stream, uint64_t i) {
  double z0, z1;
  normal_pair(stream, i >> 1, &z0, &z1);
  return (i & 1) ? z1 : z0;
}

/* Integer uniform on {-m, ..., m}. */
int64_t npg_int(uint64_t stream, uint64_t i, int64_t m) {
  uint64_t span = (uint64_t)(2 * m + 1);
  return (int64_t)((npg_draw(stream, i) >> 11) % span) - m;
}

/* ---- encodings: double -> storage bits, round to nearest even ---------- */

static inline uint32_t f32_bits(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return u;
}

/* binary32 -> bfloat16: keep the top 16 bits, rounding the low 16 to
 * nearest, ties to even.  NaN stays NaN (quiet bit forced). */
static uint16_t bf16_from_f32(float f) {
  uint32_t u = f32_bits(f);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu))
    return (uint16_t)((u >> 16) | 0x0040u);
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7FFFu + lsb;
  return (uint16_t)(u >> 16);
}

/* double -> bfloat16 with one rounding: the double is first cut to binary32
 * with round-to-odd (sticky bit), which makes the later rounding to 8
 * significand bits equal to direct rounding of the double. */
uint16_t npg_bf16(double v) {
  float f = (float)v; /* round to nearest even */
  if (isfinite(v) && (double)f != v) {
    /* redo as round-to-odd: truncate toward zero, then set the last bit */
    uint32_t u = f32_bits(f);
    double back = (double)f;
    if (fabs(back) > fabs(v)) u -= 1; /* step back toward zero */
    u |= 1u;
    memcpy(&f, &u, 4);
  }
  return bf16_from_f32(f);
}

/* double -> IEEE binary16, round to nearest even, overflow to infinity.
 * Works on the bits of the double: 52-bit fraction, 11-bit exponent. */
uint16_t npg_f16(double v) {
  uint64_t b;
  memcpy(&b, &v, 8);
  const uint16_t sign = (uint16_t)((b >> 48) & 0x8000u);
  const int ex = (int)((b >> 52) & 0x7FF);
  const uint64_t frac = b & ((1ULL << 52) - 1);
  if (ex == 0x7FF) return frac ? 0x7E00u : (uint16_t)(sign | 0x7C00u);
  const int e = ex - 1023; /* unbiased exponent of a normal double */
  if (ex == 0 || e < -25) return sign; /* below half the smallest subnormal */
  if (e > 15) return sign | 0x7C00u;
  const uint64_t sig = (1ULL << 52) | frac; /* 53-bit significand */
  int shift, exp16;
  if (e >= -14) { /* normal binary16: keep 11 significant bits */
    shift = 42;
    exp16 = e + 15;
  } else { /* subnormal binary16: units of 2^-24 */
    shift = 28 - e;
    exp16 = 0;
  }
  uint64_t m = sig >> shift;
  const uint64_t rem = sig & ((1ULL << shift) - 1), half = 1ULL << (shift - 1);
  if (rem > half || (rem == half && (m & 1u))) ++m;
  if (exp16 == 0) return sign | (uint16_t)m; /* m == 1024 is the smallest normal */
  if (m == 2048) {
    m = 1024;
    ++exp16;
  }
  if (exp16 >= 31) return sign | 0x7C00u;
  return sign | (uint16_t)((exp16 << 10) | (m - 1024));
}

static inline void put(int dtype, void* out, size_t i, double v) {
  if (dtype == NPG_F32) {
    ((float*)out)[i] = (float)v;
  } else if (dtype == NPG_F16) {
    ((uint16_t*)out)[i] = npg_f16(v);
  } else {
    ((uint16_t*)out)[i] = npg_bf16(v);
  }
}

/* ---- threaded fill ------------------------------------------------------ */

enum { KIND_RECORDS = 0, KIND_MATRIX = 1 };

typedef struct {
  int kind, dtype, dyadic;
  uint64_t seed;
  uint32_t tensor;
  int64_t layer0, layers, rows, cols;
  double scale;    /* std (gaussian) or power-of-two unit (dyadic) */
  int64_t mrange;  /* dyadic integer range */
  void* out;
  int64_t row_begin, row_end; /* rows over the flattened [layers][rows] */
} fill_job;

/* One row of `len` elements, stream indices idx0 .. idx0+len-1, written at
 * out[base ..].  Gaussian values are produced a Box-Muller pair at a time;
 * the result equals element-wise npg_normal. */
static void fill_row(const fill_job* j, uint64_t st, uint64_t idx0, int64_t len, size_t base) {
  int64_t c = 0;
  if (j->dyadic) {
    for (; c < len; ++c)
      put(j->dtype, j->out, base + (size_t)c,
          (double)npg_int(st, idx0 + (uint64_t)c, j->mrange) * j->scale);
    return;
  }
  if (idx0 & 1) { /* odd start: first element is the sine half of a pair */
    put(j->dtype, j->out, base, npg_normal(st, idx0) * j->scale);
    c = 1;
  }
  for (; c + 1 < len; c += 2) {
    double z0, z1;
    normal_pair(st, (idx0 + (uint64_t)c) >> 1, &z0, &z1);
    put(j->dtype, j->out, base + (size_t)c, z0 * j->scale);
    put(j->dtype, j->out, base + (size_t)c + 1, z1 * j->scale);
  }
  if (c < len) put(j->dtype, j->out, base + (size_t)c, npg_normal(st, idx0 + (uint64_t)c) * j->scale);
}

/* Records: element c of the gate, up or down^T row of neuron n in layer l is
 * drawn from stream (seed, tensor 1/2/3, l) at index n*d + c. */
static void* fill_worker(void* p) {
  fill_job* j = (fill_job*)p;
  for (int64_t rr = j->row_begin; rr < j->row_end; ++rr) {
    int64_t l = j->layer0 + rr / j->rows;
    int64_t n = rr % j->rows;
    if (j->kind == KIND_RECORDS) {
      int64_t d = j->cols;
      for (int part = 0; part < 3; ++part) {
        uint64_t st = npg_stream(j->seed, (uint32_t)(1 + part), (uint32_t)l);
        size_t base = (size_t)rr * 3 * d + (size_t)part * d;
        fill_row(j, st, (uint64_t)(n * d), d, base);
      }
    } else {
      uint64_t st = npg_stream(j->seed, j->tensor, (uint32_t)l);
      size_t base = (size_t)rr * j->cols;
      fill_row(j, st, (uint64_t)(n * j->cols), j->cols, base);
    }
  }
  return NULL;
}

static int run_fill(fill_job proto, int nthreads) {
  int64_t total = proto.layers * proto.rows;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  if (total < nthreads) nthreads = total > 0 ? (int)total : 1;
  pthread_t th[256];
  fill_job jobs[256];
  int started = 0;
  for (int t = 0; t < nthreads; ++t) {
    jobs[t] = proto;
    jobs[t].row_begin = total * t / nthreads;
    jobs[t].row_end = total * (t + 1) / nthreads;
    if (t == nthreads - 1) {
      fill_worker(&jobs[t]);
    } else if (pthread_create(&th[t], NULL, fill_worker, &jobs[t]) == 0) {
      ++started;
    } else {
      fill_worker(&jobs[t]);
      th[t] = 0;
    }
  }
  for (int t = 0; t < nthreads - 1; ++t)
    if (th[t]) pthread_join(th[t], NULL);
  (void)started;
  return 0;
}

/* MLP neuron records of layers [layer0, layer0+layers), written to `out`
 * as [layers][F][3d].  Gaussian N(0, std^2), or dyadic m * unit with m
 * uniform on {-mrange..mrange} when dyadic != 0. */
int npg_fill_records(int dtype, uint64_t seed, int64_t layer0, int64_t layers,
                     int64_t F, int64_t d, int dyadic, double std_or_unit,
                     int64_t mrange, void* out, int nthreads) {
  fill_job j;
  memset(&j, 0, sizeof j);
  j.kind = KIND_RECORDS;
  j.dtype = dtype;
  j.dyadic = dyadic;
  j.seed = seed;
  j.layer0 = layer0;
  j.layers = layers;
  j.rows = F;
  j.cols = d;
  j.scale = std_or_unit;
  j.mrange = mrange;
  j.out = out;
  return run_fill(j, nthreads);
}

/* A [layers][rows][cols] matrix stack for tensor id `tensor` (4 = predictor
 * A, 5 = predictor B), element (l, i, c) from stream (seed, tensor, l) at
 * index i*cols + c. */
int npg_fill_matrix(int dtype, uint64_t seed, uint32_t tensor, int64_t layer0,
                    int64_t layers, int64_t rows, int64_t cols, int dyadic,
                    double std_or_unit, int64_t mrange, void* out,
                    int nthreads) {
  fill_job j;
  memset(&j, 0, sizeof j);
  j.kind = KIND_MATRIX;
  j.dtype = dtype;
  j.dyadic = dyadic;
  j.seed = seed;
  j.tensor = tensor;
  j.layer0 = layer0;
  j.layers = layers;
  j.rows = rows;
  j.cols = cols;
  j.scale = std_or_unit;
  j.mrange = mrange;
  j.out = out;
  return run_fill(j, nthreads);
}

/* Hidden states h_0..h_{T-1}, [T][d], encoded as `dtype`.
 * Gaussian: h_0 = e_0, h_t = rho*h_{t-1} + sqrt(1-rho^2)*e_t with
 * e_t[c] = N(0,1) from stream (seed, 6, t) at index c; kept in double.
 * Dyadic (dyadic != 0): h_0[c] uniform on {-mrange..mrange}; afterwards each
 * coordinate is redrawn with probability `rho` (read as a redraw rate) and
 * kept otherwise. */
int npg_hidden(int dtype, uint64_t seed, int64_t T, int64_t d, double rho,
               int dyadic, int64_t mrange, void* out, double* out_f64) {
  double prev_scale = rho, fresh_scale = sqrt(1.0 - rho * rho);
  for (int64_t c = 0; c < d; ++c) {
    double h = 0.0;
    for (int64_t t = 0; t < T; ++t) {
      uint64_t st = npg_stream(seed, 6, (uint32_t)t);
      if (dyadic) {
        uint64_t st_pick = npg_stream(seed, 7, (uint32_t)t);
        double r = unit_open(npg_draw(st_pick, (uint64_t)c));
        if (t == 0 || r < rho) h = (double)npg_int(st, (uint64_t)c, mrange);
      } else {
        double e = npg_normal(st, (uint64_t)c);
        h = (t == 0) ? e : prev_scale * h + fresh_scale * e;
      }
      put(dtype, out, (size_t)(t * d + c), h);
      if (out_f64) out_f64[t * d + c] = h;
    }
  }
  return 0;
}

/* The centroid predictor's feature vectors f_0..f_{T-1}, [T][D], the same
 * AR(1) recursion as the hidden states on stream (seed, 20, t). */
int npg_features(int dtype, uint64_t seed, int64_t T, int64_t D, double rho, void* out) {
  double prev_scale = rho, fresh_scale = sqrt(1.0 - rho * rho);
  for (int64_t c = 0; c < D; ++c) {
    double f = 0.0;
    for (int64_t t = 0; t < T; ++t) {
      double e = npg_normal(npg_stream(seed, 20, (uint32_t)t), (uint64_t)c);
      f = (t == 0) ? e : prev_scale * f + fresh_scale * e;
      put(dtype, out, (size_t)(t * D + c), f);
    }
  }
  return 0;
}

/* Centroid mask bank [2][L][K][W] (W = ceil(F/32) words, bit n%32 of word
 * n/32; gate masks, then up masks).  Neuron n of layer l is "hot" (for both
 * projections) when a uniform draw of stream (seed, 21, l) at index n is
 * below q_hot; bit n of centroid c of projection p is set when a uniform draw
 * of stream (seed, 23 + p, l) at index c*F + n is below p_hot (hot) or
 * p_cold (not). */
typedef struct {
  uint64_t seed;
  int64_t L, K, F;
  double q_hot, p_hot, p_cold;
  uint32_t* out;
  int next, total;
  pthread_mutex_t mu;
} bank_job;

static void* bank_worker(void* arg) {
  bank_job* j = (bank_job*)arg;
  const int64_t W = (j->F + 31) / 32;
  for (;;) {
    pthread_mutex_lock(&j->mu);
    int pl = j->next++;
    pthread_mutex_unlock(&j->mu);
    if (pl >= j->total) return NULL;
    const int p = (int)(pl / j->L);
    const int64_t l = pl % j->L;
    uint64_t st_hot = npg_stream(j->seed, 21, (uint32_t)l);
    uint64_t st_bit = npg_stream(j->seed, 23 + (uint32_t)p, (uint32_t)l);
    for (int64_t c = 0; c < j->K; ++c) {
      uint32_t* m = j->out + ((size_t)pl * j->K + c) * W;
      memset(m, 0, sizeof(uint32_t) * (size_t)W);
      for (int64_t n = 0; n < j->F; ++n) {
        const int hot = unit_open(npg_draw(st_hot, (uint64_t)n)) < j->q_hot;
        const double u = unit_open(npg_draw(st_bit, (uint64_t)(c * j->F + n)));
        if (u < (hot ? j->p_hot : j->p_cold)) m[n >> 5] |= 1u << (n & 31);
      }
    }
  }
}

int npg_fill_bank(uint64_t seed, int64_t L, int64_t K, int64_t F, double q_hot, double p_hot,
                  double p_cold, uint32_t* out, int nthreads) {
  bank_job j;
  j.seed = seed; j.L = L; j.K = K; j.F = F;
  j.q_hot = q_hot; j.p_hot = p_hot; j.p_cold = p_cold;
  j.out = out; j.next = 0; j.total = (int)(2 * L);
  pthread_mutex_init(&j.mu, NULL);
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 64) nthreads = 64;
  pthread_t th[64];
  int started = 0;
  for (int t = 0; t < nthreads; ++t)
    if (pthread_create(&th[t], NULL, bank_worker, &j) == 0) ++started;
  if (started == 0) bank_worker(&j);
  for (int t = 0; t < started; ++t) pthread_join(th[t], NULL);
  pthread_mutex_destroy(&j.mu);
  return 0;
}

/* Encode an array of doubles (tests use this to build small inputs). */
void npg_encode(int dtype, const double* in, int64_t n, void* out) {
  for (int64_t i = 0; i < n; ++i) put(dtype, out, (size_t)i, in[i]);
}
