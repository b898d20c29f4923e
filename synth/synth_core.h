/*
 * synth_core.h -- seeded synthetic-gradient recipe shared by the host (C) and
 * device (HIP) fills.  Input generation only: nothing here is part of the
 * compressor's arithmetic.
 *
 * Every value is a deterministic function of (seed, step t, worker i,
 * coordinate j).  Only integer operations and correctly rounded binary32
 * add / sub / mul / fmaf are used (no libm), so a host build and a device
 * build produce identical bits.  Both must be compiled with
 * -ffp-contract=off and without fast-math.
 *
 * Random bits: a counter hash built on the SplitMix64 mixing function
 * (Steele, Lea & Flood, OOPSLA 2014).  Normals: Box-Muller (1958) with
 * polynomial ln / sin / cos written out below.  Student-t(3): z0 / sqrt(chi2_3
 * / 3) from four normals.
 */
#ifndef SYNTH_CORE_H
#define SYNTH_CORE_H
#include <stdint.h>

#if defined(__HIPCC__)
#define SYNTH_FN __host__ __device__ static inline
#else
#include <math.h>
#define SYNTH_FN static inline
#endif

typedef struct {
  int32_t family;     /* 0: scale * (m_j + noise * e_ij);  1: Student-t mix  */
  int32_t out_bf16;   /* 0: binary32 output; 1: bf16 (round to nearest even) */
  int64_t d;          /* coordinates per worker                               */
  int32_t N;          /* workers                                              */
  int32_t per_coord;  /* 1: scale[] has d entries; 0: one per segment         */
  uint64_t seed;      /* data seed                                            */
  float noise;        /* family 0: weight of the per-worker normal            */
  float c_shared;     /* family 1: weight of the shared Student-t draw        */
  float c_own;        /* family 1: weight of the per-worker Student-t draw    */
  float boost;        /* factor for boosted coordinates                       */
  uint32_t boost_threshold; /* coordinate j boosted if hi32(bits) < this; 0 off */
  int32_t nseg;       /* number of segments (per_coord == 0)                  */
  const int64_t *seg_begin; /* [nseg] first coordinate of each segment, [0]=0 */
  const float *scale;       /* [nseg] or [d]                                  */
} synth_plan;

enum { SYNTH_STREAM_SHARED = 1, SYNTH_STREAM_OWN = 2, SYNTH_STREAM_BOOST = 3 };

SYNTH_FN uint64_t synth_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

/* Key of one random stream: (seed, stream id, step, worker). */
SYNTH_FN uint64_t synth_key(uint64_t seed, uint64_t stream, uint64_t t,
                            uint64_t i) {
  uint64_t k = synth_mix64(seed + 0x9E3779B97F4A7C15ull);
  k = synth_mix64(k + stream * 0xD1B54A32D192ED03ull);
  k = synth_mix64(k + t * 0x8CB92BA72F3D8DD7ull);
  return synth_mix64(k + i * 0xABC98388FB8FAC03ull);
}

SYNTH_FN uint64_t synth_bits(uint64_t key, uint64_t ctr) {
  return synth_mix64(key + (ctr + 1ull) * 0x9E3779B97F4A7C15ull);
}

SYNTH_FN float synth_f32(uint32_t b) {
  float f;
  __builtin_memcpy(&f, &b, 4);
  return f;
}

SYNTH_FN uint32_t synth_u32(float f) {
  uint32_t b;
  __builtin_memcpy(&b, &f, 4);
  return b;
}

/* ln(u) for u in (0, 1]: u = 2^e f with f in [sqrt(1/2), sqrt(2)), then the
 * Taylor series of ln(1 + t), t = f - 1, to degree 18 (|t| <= 0.4143,
 * truncation error < 3e-9). */
SYNTH_FN float synth_log(float u) {
  uint32_t b = synth_u32(u);
  int32_t e = (int32_t)(b >> 23) - 127;
  float f = synth_f32((b & 0x007FFFFFu) | 0x3F800000u);
  if (f > 1.41421354f) {
    f = f * 0.5f;
    e = e + 1;
  }
  const float t = f - 1.0f;
  /* (-1)^(k+1) / k for k = 1..18, folded to binary32 at compile time */
  const float ck[18] = {1.0f,         -1.0f / 2.0f,  1.0f / 3.0f,  -1.0f / 4.0f,
                        1.0f / 5.0f,  -1.0f / 6.0f,  1.0f / 7.0f,  -1.0f / 8.0f,
                        1.0f / 9.0f,  -1.0f / 10.0f, 1.0f / 11.0f, -1.0f / 12.0f,
                        1.0f / 13.0f, -1.0f / 14.0f, 1.0f / 15.0f, -1.0f / 16.0f,
                        1.0f / 17.0f, -1.0f / 18.0f};
  float p = 0.0f;
  for (int k = 17; k >= 0; --k) p = fmaf(p, t, ck[k]);
  return fmaf((float)e, 0.693147182f, p * t);
}

/* sin and cos of 2*pi*u for u in [0, 1): quarter-turn reduction (exact), then
 * Taylor series on [0, pi/2) to degree 13 (sin) and 14 (cos). */
SYNTH_FN void synth_sincos_turn(float u, float *s_out, float *c_out) {
  const float x = u * 4.0f;
  const int32_t q = (int32_t)x;
  const float y = x - (float)q;
  const float phi = y * 1.57079637f;
  const float p2 = phi * phi;
  float s = 0.0f, c = 0.0f;
  /* sin(phi)/phi = sum_k (-1)^k p2^k / (2k+1)!,  k = 0..6 */
  {
    const float cs[7] = {1.0f, -1.0f / 6.0f, 1.0f / 120.0f, -1.0f / 5040.0f,
                         1.0f / 362880.0f, -1.0f / 39916800.0f,
                         1.0f / 6227020800.0f};
    for (int k = 6; k >= 0; --k) s = fmaf(s, p2, cs[k]);
    s = s * phi;
  }
  /* cos(phi) = sum_k (-1)^k p2^k / (2k)!,  k = 0..7 */
  {
    const float cc[8] = {1.0f, -0.5f, 1.0f / 24.0f, -1.0f / 720.0f,
                         1.0f / 40320.0f, -1.0f / 3628800.0f,
                         1.0f / 479001600.0f, -1.0f / 87178291200.0f};
    for (int k = 7; k >= 0; --k) c = fmaf(c, p2, cc[k]);
  }
  switch (q & 3) {
    case 0: *s_out = s; *c_out = c; break;
    case 1: *s_out = c; *c_out = -s; break;
    case 2: *s_out = -s; *c_out = -c; break;
    default: *s_out = -c; *c_out = s; break;
  }
}

/* 1/sqrt(x) for normal x > 0: bit-level first guess (Lomont, "Fast inverse
 * square root", 2003) and four Newton steps. */
SYNTH_FN float synth_rsqrt(float x) {
  float y = synth_f32(0x5F3759DFu - (synth_u32(x) >> 1));
  const float hx = 0.5f * x;
  for (int k = 0; k < 4; ++k) {
    const float yy = y * y;
    y = y * fmaf(-hx, yy, 1.5f);
  }
  return y;
}

/* Two independent N(0,1) draws from 64 random bits (Box-Muller). */
SYNTH_FN void synth_normal2(uint64_t bits, float *za, float *zb) {
  const uint32_t k1 = (uint32_t)(bits >> 40);
  const uint32_t k2 = (uint32_t)(bits >> 16) & 0x00FFFFFFu;
  const float u1 = (float)(k1 + 1u) * 0x1.0p-24f; /* (0, 1], exact */
  const float u2 = (float)k2 * 0x1.0p-24f;        /* [0, 1),  exact */
  const float x = -2.0f * synth_log(u1);
  const float R = (x > 0.0f) ? x * synth_rsqrt(x) : 0.0f;
  float s, c;
  synth_sincos_turn(u2, &s, &c);
  *za = R * c;
  *zb = R * s;
}

SYNTH_FN float synth_normal(uint64_t key, uint64_t ctr) {
  float a, b;
  synth_normal2(synth_bits(key, ctr), &a, &b);
  return a;
}

/* Student-t with 3 degrees of freedom: z0 / sqrt((z1^2 + z2^2 + z3^2) / 3). */
SYNTH_FN float synth_student3(uint64_t key, uint64_t j) {
  float z0, z1, z2, z3;
  synth_normal2(synth_bits(key, 2u * j), &z0, &z1);
  synth_normal2(synth_bits(key, 2u * j + 1u), &z2, &z3);
  float chi = z1 * z1;
  chi = fmaf(z2, z2, chi);
  chi = fmaf(z3, z3, chi);
  chi = chi * 0.333333343f;
  if (chi < 1.0e-30f) chi = 1.0e-30f;
  return z0 * synth_rsqrt(chi);
}

SYNTH_FN float synth_scale_at(const synth_plan *pl, int64_t j) {
  if (pl->per_coord) return pl->scale[j];
  int32_t lo = 0, hi = pl->nseg; /* last segment whose begin <= j */
  while (hi - lo > 1) {
    const int32_t mid = (lo + hi) >> 1;
    if (pl->seg_begin[mid] <= j) lo = mid; else hi = mid;
  }
  return pl->scale[lo];
}

/* Keys for one step and worker. */
typedef struct {
  uint64_t shared, own, boost;
} synth_keys;

SYNTH_FN synth_keys synth_step_keys(const synth_plan *pl, int64_t t,
                                    int32_t i) {
  synth_keys k;
  k.shared = synth_key(pl->seed, SYNTH_STREAM_SHARED, (uint64_t)t, 0u);
  k.own = synth_key(pl->seed, SYNTH_STREAM_OWN, (uint64_t)t, (uint64_t)i);
  k.boost = synth_key(pl->seed, SYNTH_STREAM_BOOST, 0u, 0u);
  return k;
}

/* Gradient value of worker i at coordinate j (binary32). */
SYNTH_FN float synth_value(const synth_plan *pl, const synth_keys *k,
                           int64_t j) {
  float s = synth_scale_at(pl, j);
  if (pl->boost_threshold != 0u &&
      (uint32_t)(synth_bits(k->boost, (uint64_t)j) >> 32) < pl->boost_threshold)
    s = pl->boost * s;
  if (pl->family == 0) {
    const float mj = synth_normal(k->shared, (uint64_t)j);
    const float eij = synth_normal(k->own, (uint64_t)j);
    return s * fmaf(pl->noise, eij, mj);
  }
  const float tj = synth_student3(k->shared, (uint64_t)j);
  const float tij = synth_student3(k->own, (uint64_t)j);
  return s * fmaf(pl->c_shared, tj, pl->c_own * tij);
}

/* binary32 -> bf16 bits, round to nearest even (finite inputs). */
SYNTH_FN uint16_t synth_to_bf16(float v) {
  uint32_t b = synth_u32(v);
  b = b + 0x7FFFu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}

#endif
