/*
 * Seeded synthetic logits for the drafter-evaluation workloads.
 *
 * This file is input plumbing only: it draws numbers and rounds them to the
 * storage type. It contains none of the arithmetic of the method being tested
 * (no softmax, no acceptance probability, no learner). Both the oracle and the
 * GPU path consume the bytes it writes.
 *
 * Generator (counter based, so any row can be produced on its own):
 *   mix64      : the splitmix64 output finaliser (Steele, Lea, Flood 2014).
 *   row key    : mix64-chained over (seed, round, tensor, query b, position k).
 *   element v  : two 64-bit draws h1 = mix64(key + (2v+1)*G), h2 = mix64(key + (2v+2)*G),
 *                G = 0x9E3779B97F4A7C15. Their eight 16-bit fields c_j are
 *                summed; Z = (sum c_j - 262140) * sqrt(1.5) / 65536 is the
 *                standardised Irwin-Hall(8) variate (mean 0, variance 1,
 *                support +-4.9). It needs only integer work plus one fp64
 *                multiply, so it is bit-reproducible on any IEEE machine.
 *   target     : t = sigma_t * Z (+ boost on nboost distinct seeded indices of
 *                the row), rounded to the storage type.
 *   drafter i  : d = decode(stored t) + s * Z_i, rounded (the noise is added to
 *                exactly what the kernel reads).
 *   rounding   : fp64 -> fp32 round-to-nearest-even, then (bf16 storage)
 *                fp32 -> bf16 round-to-nearest-even on the bit pattern, or (fp16
 *                storage) fp32 -> IEEE binary16 round-to-nearest-even, with
 *                gradual underflow and overflow to infinity.
 * Build with -ffp-contract=off so that no multiply-add is fused.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

#define SYN_F32 0
#define SYN_BF16 1
#define SYN_F16 2

static const uint64_t GOLD = 0x9E3779B97F4A7C15ULL;

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static inline uint64_t chain(uint64_t key, uint64_t x) { return mix64(key ^ mix64(x + GOLD)); }

uint64_t synth_row_key(uint64_t seed, int64_t round, int64_t tensor, int64_t b, int64_t k) {
  uint64_t h = mix64(seed + GOLD);
  h = chain(h, (uint64_t)round);
  h = chain(h, (uint64_t)tensor);
  h = chain(h, (uint64_t)b);
  h = chain(h, (uint64_t)k);
  return h;
}

static inline double normal_at(uint64_t key, int64_t v) {
  uint64_t h1 = mix64(key + (uint64_t)(2 * v + 1) * GOLD);
  uint64_t h2 = mix64(key + (uint64_t)(2 * v + 2) * GOLD);
  int64_t s = 0;
  for (int j = 0; j < 4; ++j) {
    s += (int64_t)((h1 >> (16 * j)) & 0xFFFF);
    s += (int64_t)((h2 >> (16 * j)) & 0xFFFF);
  }
  return (double)(s - 262140) * (1.2247448713915890491 / 65536.0);
}

double synth_normal(uint64_t key, int64_t v) { return normal_at(key, v); }

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static inline float bf16_to_f32(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

/* fp32 -> IEEE 754 binary16 (1 sign, 5 exponent, 10 fraction bits, bias 15), round to
   nearest, ties to even. */
static inline uint16_t f32_to_f16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  const uint32_t sign = (u >> 16) & 0x8000u;
  const uint32_t a = u & 0x7FFFFFFFu;
  if (a > 0x7F800000u) return (uint16_t)(sign | 0x7E00u); /* NaN: a quiet NaN */
  if (a >= 0x477FF000u) return (uint16_t)(sign | 0x7C00u); /* >= 65520 rounds to infinity */
  const int e = (int)(a >> 23) - 127;
  const uint32_t sig = (a & 0x7FFFFFu) | 0x800000u; /* 24-bit significand (normal inputs) */
  if (e >= -14) {                                    /* a binary16 normal */
    uint32_t h = ((uint32_t)(e + 15) << 10) | ((a & 0x7FFFFFu) >> 13);
    const uint32_t rem = a & 0x1FFFu;
    if (rem > 0x1000u || (rem == 0x1000u && (h & 1u))) h += 1u; /* a carry moves the exponent */
    return (uint16_t)(sign | h);
  }
  /* a binary16 subnormal m 2^-24: m = sig 2^(e + 1), rounded */
  const int sh = -(e + 1);
  if (sh >= 32) return (uint16_t)sign; /* below 2^-32: rounds to zero */
  uint32_t m = sig >> sh;
  const uint32_t rem = sig & ((1u << sh) - 1u), half = 1u << (sh - 1);
  if (rem > half || (rem == half && (m & 1u))) m += 1u; /* 1024 is the smallest normal */
  return (uint16_t)(sign | m);
}

static inline float f16_to_f32(uint16_t h) {
  const uint32_t sign = (uint32_t)(h & 0x8000u) << 16;
  const uint32_t ex = (h >> 10) & 0x1Fu, m = h & 0x3FFu;
  float f;
  if (ex == 0) {
    f = ldexpf((float)m, -24);
    if (sign) f = -f;
    return f;
  }
  const uint32_t u = ex == 0x1Fu ? (sign | 0x7F800000u | (m << 13)) : (sign | ((ex + 112u) << 23) | (m << 13));
  memcpy(&f, &u, 4);
  return f;
}

/* The binary16 bit pattern of an fp64 value as the generator stores it (fp32 first). */
uint16_t synth_round_f16(double x) { return f32_to_f16_rne((float)x); }

/* Round an fp64 value to the storage type; returns the stored value decoded back. */
static inline double store_one(double x, int dtype, void* out, int64_t idx) {
  float f = (float)x;
  if (dtype == SYN_F32) {
    ((float*)out)[idx] = f;
    return (double)f;
  }
  if (dtype == SYN_F16) {
    uint16_t h = f32_to_f16_rne(f);
    ((uint16_t*)out)[idx] = h;
    return (double)f16_to_f32(h);
  }
  uint16_t h = f32_to_bf16_rne(f);
  ((uint16_t*)out)[idx] = h;
  return (double)bf16_to_f32(h);
}

static int cmp_i64(const void* a, const void* b) {
  const int64_t x = *(const int64_t*)a, y = *(const int64_t*)b;
  return (x > y) - (x < y);
}

/* nboost distinct indices in [0, V), drawn by hashing with rejection of repeats. */
int synth_boost_indices(uint64_t seed, int64_t round, int64_t b, int64_t k, int64_t V, int nboost,
                        int64_t* idx) {
  if (nboost > V) return -1;
  uint64_t key = synth_row_key(seed, round, 0x626F6F7374LL /* "boost" */, b, k);
  int n = 0;
  for (uint64_t ctr = 0; n < nboost; ++ctr) {
    int64_t cand = (int64_t)(mix64(key + (ctr + 1) * GOLD) % (uint64_t)V);
    int dup = 0;
    for (int j = 0; j < n; ++j) dup |= (idx[j] == cand);
    if (!dup) idx[n++] = cand;
  }
  return 0;
}

/*
 * Fill rows of the [R][B][K][V] logits tensor, R = N + 1 (row 0 = target,
 * row 1 + i = drafter i).
 *   rows      : tensor rows to produce (values in [0, N]), nrows of them.
 *   bk        : (b, k) pairs to produce, nbk of them (b-major pairs), or NULL for all B*K in order.
 *   scale     : [B][N] noise scale of drafter i at query b.
 *   out       : [nrows][nbk][ld] elements of the storage type; only the first V of each row are written.
 */
int synth_fill(int dtype, int64_t V, int64_t ld, int B, int K, int N, uint64_t seed, int64_t round,
               double sigma_t, int nboost, double boost, const double* scale, const int32_t* rows,
               int nrows, const int32_t* bk, int64_t nbk, void* out) {
  if (dtype != SYN_F32 && dtype != SYN_BF16 && dtype != SYN_F16) return -1;
  if (V < 1 || ld < V || B < 1 || K < 1 || N < 1 || nboost < 0 || nboost > V) return -2;
  int64_t nitems = (bk ? nbk : (int64_t)B * K);
  int fail = 0;
  /* one (b, k) item per task: its target row once (fp64 before rounding), then every
     requested row of the item from it */
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t p = 0; p < nitems; ++p) {
    int64_t b = bk ? bk[2 * p] : p / K;
    int64_t k = bk ? bk[2 * p + 1] : p % K;
    uint64_t tkey = synth_row_key(seed, round, 0, b, k);
    double* tv = (double*)malloc(sizeof(double) * (size_t)V);
    if (!tv) {
#pragma omp atomic write
      fail = 1;
      continue;
    }
    int64_t bidx[65];
    int nb = nboost < 64 ? nboost : 64;
    if (nb > 0) synth_boost_indices(seed, round, b, k, V, nb, bidx);
    /* the indices are distinct: walk them in increasing order beside v */
    qsort(bidx, (size_t)nb, sizeof(int64_t), cmp_i64);
    bidx[nb] = V;
    int nxt = 0;
    for (int64_t v = 0; v < V; ++v) {
      double t = sigma_t * normal_at(tkey, v);
      if (bidx[nxt] == v) {
        t = t + boost;
        ++nxt;
      }
      tv[v] = t;
    }
    for (int ri = 0; ri < nrows; ++ri) {
      int row = rows[ri];
      int64_t base = ((int64_t)ri * nitems + p) * ld;
      if (row == 0) {
        for (int64_t v = 0; v < V; ++v) store_one(tv[v], dtype, out, base + v);
      } else {
        double s = scale[b * N + (row - 1)];
        uint64_t dkey = synth_row_key(seed, round, row, b, k);
        float tmpf;
        uint16_t tmph;
        for (int64_t v = 0; v < V; ++v) {
          double ts = (dtype == SYN_F32) ? store_one(tv[v], dtype, &tmpf, 0)
                                         : store_one(tv[v], dtype, &tmph, 0);
          double d = ts + s * normal_at(dkey, v);
          store_one(d, dtype, out, base + v);
        }
      }
    }
    free(tv);
  }
  return fail ? -3 : 0;
}

/* Seeded Fisher-Yates shuffle of 0..n-1 keyed by (seed, tag, b). */
void synth_permutation(uint64_t seed, int64_t tag, int64_t b, int n, int32_t* perm) {
  uint64_t key = synth_row_key(seed, 0, tag, b, 0);
  for (int i = 0; i < n; ++i) perm[i] = i;
  for (int i = n - 1; i > 0; --i) {
    int j = (int)(mix64(key + (uint64_t)(i + 1) * GOLD) % (uint64_t)(i + 1));
    int32_t t = perm[i];
    perm[i] = perm[j];
    perm[j] = t;
  }
}

/* Uniform integer in [0, n) keyed by (seed, tag, a, c); used for seeded tree descents. */
int64_t synth_uniform_int(uint64_t seed, int64_t tag, int64_t a, int64_t c, int64_t n) {
  uint64_t key = synth_row_key(seed, 0, tag, a, c);
  return (int64_t)(mix64(key + GOLD) % (uint64_t)n);
}
