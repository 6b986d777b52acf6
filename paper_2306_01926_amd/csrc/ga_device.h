// Device helpers shared by the gfx950 kernel files: bf16 conversions, the
// canonical |r|^2 split, the MFMA 32x32x16 scoring of 32 keys against blocks of
// 32 groups with the packed top-2 reduction, and the exact fp64 argmin used for
// keys whose MFMA decision is not certified.  Included inside
// namespace ga { namespace { ... } } by each kernel file.
#pragma once

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef double f64x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }
// Round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

// Storage-dtype traits: load as float, representative rounding, store.
struct F32 {
  using T = float;
  __device__ static float load(const float* p, int64_t i) { return p[i]; }
  __device__ static float rep(float c) { return c; }
  __device__ static void store(float* p, int64_t i, float r) { p[i] = r; }
};
struct BF16 {
  using T = uint16_t;
  __device__ static float load(const uint16_t* p, int64_t i) { return bf16_to_f32(p[i]); }
  __device__ static float rep(float c) { return bf16_to_f32(f32_to_bf16(c)); }
  __device__ static void store(uint16_t* p, int64_t i, float r) { p[i] = (uint16_t)(__float_as_uint(r) >> 16); }
};

// min / max of finite scores as a median of three with -FLT_MAX / FLT_MAX:
// one v_med3_f32 each, without the NaN canonicalisation fminf / fmaxf need.
__device__ __forceinline__ float min2(float a, float b) { return __builtin_amdgcn_fmed3f(a, b, -FLT_MAX); }
__device__ __forceinline__ float max2(float a, float b) { return __builtin_amdgcn_fmed3f(a, b, FLT_MAX); }

// v_min3_f32 without the NaN canonicalisation the compiler adds around
// fminf-based min3 (the operands are finite scores).
__device__ __forceinline__ float min3f(float a, float b, float c) {
  float r;
  asm("v_min3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

__device__ __forceinline__ float readlane_f(float x, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}

// |r|^2 as an fp64 fma chain over c = 0..63 (lane c holds r_c); same value in all lanes.
__device__ double canon_nrm_wave(float r) {
  double acc = 0.0;
#pragma unroll 8
  for (int c = 0; c < 64; ++c) {
    const double rc = (double)readlane_f(r, c);
    acc = fma(rc, rc, acc);
  }
  return acc;
}

// |r|^2 as three bf16 terms hi + mid + lo (each the bf16 rounding of the
// remainder; the two subtractions are exact), |sum - nrm| <= ~2^-24 nrm.  The
// assign kernel adds them to the scores through one extra MFMA k-step.
__device__ void write_nsplit(double nrm, uint16_t* dst) {
  const uint32_t hi = f32_to_bf16((float)nrm);
  const double r1 = nrm - (double)bf16_to_f32(hi);
  const uint32_t mid = f32_to_bf16((float)r1);
  const double r2 = r1 - (double)bf16_to_f32(mid);
  const uint32_t lo = f32_to_bf16((float)r2);
  *(u32x4*)dst = u32x4{hi | (mid << 16), lo, 0u, 0u};
}


// The assign kernel's LDS copy of -2R stores 16-byte chunk c of row r at chunk
// c ^ ((r >> 1) & 7) of a 128-byte row: 16 consecutive rows reading the same
// logical chunk then hit 16 distinct groups of 4 banks (no padding needed).
__device__ __forceinline__ int swz(int r, int c) { return r * 64 + 8 * (c ^ ((r >> 1) & 7)); }

// Exact assignment of NK bf16 keys at once by a whole wave, the
// representatives read from the LDS copy of -2R.  Same definition as
// exact_argmin_wave (score fma(-2, k.r, |r|^2) with k.r an fp64 fma chain over
// c = 0..63, lowest index among minima): x = -2r is exact in bf16 and every
// partial sum of the chain over k_c x_c is exactly -2 times the one over
// k_c r_c (the partial sums stay far from the fp64 subnormal range), so the
// score is |r|^2 + (chain over k_c x_c) with one rounding.  kd: the keys as
// fp64 rows [NK][64] in LDS (the same words in every lane).  Lane l takes
// groups l, l + 64, l + 128, ... in ascending order, two at a time, and each
// converts its representatives' features once for all NK keys.
template <int NK>
__device__ void exact_argmin_keys(const double* kd, const uint16_t* Rs, const double* __restrict__ nrm, int N,
                                  int* jb) {
  const int lane = threadIdx.x & 63;
  double best[NK];
  int bj[NK];
#pragma unroll
  for (int b = 0; b < NK; ++b) {
    best[b] = INFINITY;
    bj[b] = 0x7fffffff;
  }
  for (int j0 = lane; j0 < N; j0 += 128) {
    const int j1 = j0 + 64;
    const bool two = j1 < N;
    const int j1r = two ? j1 : j0;  // a row that exists
    const double n0 = nrm[j0], n1 = nrm[j1r];  // in flight during the dot products
    double d0[NK], d1[NK];
#pragma unroll
    for (int b = 0; b < NK; ++b) d0[b] = d1[b] = 0.0;
#pragma unroll 2
    for (int i = 0; i < 8; ++i) {
      const u32x4 w0 = *(const u32x4*)(Rs + swz(j0, i)), w1 = *(const u32x4*)(Rs + swz(j1r, i));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double x0 = (double)bf16_to_f32(w0[e] & 0xffffu), y0 = (double)bf16_to_f32(w0[e] >> 16);
        const double x1 = (double)bf16_to_f32(w1[e] & 0xffffu), y1 = (double)bf16_to_f32(w1[e] >> 16);
#pragma unroll
        for (int b = 0; b < NK; ++b) {
          const f64x2 kk = *(const f64x2*)(kd + b * 64 + 8 * i + 2 * e);
          d0[b] = fma(kk[0], x0, d0[b]);
          d0[b] = fma(kk[1], y0, d0[b]);
          d1[b] = fma(kk[0], x1, d1[b]);
          d1[b] = fma(kk[1], y1, d1[b]);
        }
      }
    }
#pragma unroll
    for (int b = 0; b < NK; ++b) {
      const double s0 = n0 + d0[b];
      if (s0 < best[b]) {
        best[b] = s0;
        bj[b] = j0;
      }
      const double s1 = n1 + d1[b];
      if (two && s1 < best[b]) {
        best[b] = s1;
        bj[b] = j1;
      }
    }
  }
#pragma unroll
  for (int b = 0; b < NK; ++b) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const double ob = __shfl_xor(best[b], off);
      const int oj = __shfl_xor(bj[b], off);
      if (ob < best[b] || (ob == best[b] && oj < bj[b])) {
        best[b] = ob;
        bj[b] = oj;
      }
    }
    jb[b] = bj[b];
  }
}

// Scores are ranked as packed floats: the low 4 mantissa bits of a score are
// replaced by its accumulator register index v (0..15), so one min/med3 chain
// keeps value and register of the best two.  The block of the best is tracked
// beside it and the lane half is resolved when the halves merge, so the
// group of a packed best (v, block b, half h) is 32 b + 8 (v/4) + 4 h + v%4.
constexpr uint32_t kPackMask = 15u;

// Top-2 of one block's 16 scores folded into the running (M1, M2, B1 = block
// of M1).  Over quads: with m1 <= m2 the two smallest so far and
// a = min3(m1, x0, x1), the two smallest of {m1, m2, x0, x1, x2, x3} are
// min3(a, x2, x3) and min3(m2, med3(m1, x0, x1), med3(a, x2, x3)).  A packed
// value equal to M1 from a later block keeps the earlier block; such a key is
// never certified (its gap is 0), so the choice does not matter.
__device__ __forceinline__ void reduce_block(const f32x16& acc, int blk, float& M1, float& M2, int& B1) {
  const float prev = M1;
#pragma unroll
  for (int v = 0; v < 16; v += 4) {
    float x[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      x[e] = __uint_as_float((__float_as_uint(acc[v + e]) & ~kPackMask) | (uint32_t)(v + e));
    const float t01 = __builtin_amdgcn_fmed3f(M1, x[0], x[1]);
    const float a = min3f(M1, x[0], x[1]);
    const float t23 = __builtin_amdgcn_fmed3f(a, x[2], x[3]);
    M1 = min3f(a, x[2], x[3]);
    M2 = min3f(M2, t01, t23);
  }
  B1 = M1 < prev ? blk : B1;
}

// Bounds shared by every tile of a slice: the largest |r|^2 and |r| (with
// margins for their fp32 evaluation) and the error constants of the launch.
struct Certify {
  float nmaxf, rmaxf, cm, cp;
};

// (value of lane q, value of lane q + 32) in every lane l, q = l % 32.
__device__ __forceinline__ u32x2 halves(uint32_t x) {
  const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return u32x2{r[0], r[1]};
}

// Upper bound of |k| for the key whose 64 bf16 features are split over lanes
// q and q + 32 (32 each, as MFMA fragments); the same value in both lanes.
__device__ __forceinline__ float key_norm_bound(const u32x4 (&f)[4]) {
  float ss = 0.f;
#pragma unroll
  for (int s2 = 0; s2 < 4; ++s2)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = bf16_to_f32(f[s2][e] & 0xffffu), hi = bf16_to_f32(f[s2][e] >> 16);
      ss = fmaf(lo, lo, ss);
      ss = fmaf(hi, hi, ss);
    }
  const u32x2 p = halves(__float_as_uint(ss));
  return sqrtf(__uint_as_float(p[0]) + __uint_as_float(p[1])) * (1.0f + 0x1p-16f);
}

// Append this lane's entry if `mine`; the region's count `n` is wave-uniform.
__device__ __forceinline__ void wave_append(bool mine, uint32_t rec, uint32_t* region, int& n) {
  const uint64_t mask = __ballot(mine);
  if (mine)
    region[n + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u))] =
        rec;
  n += (int)__popcll(mask);
}

// The |r|^2 part of every score: block b's MFMA of the split row (A) with
// ones in the first three k slots of lanes h = 0 (B), the same for every tile.
template <int NB>
__device__ __forceinline__ void norm_terms(const u32x4 (&an)[NB], const u32x4& ones, f32x16 (&nacc)[NB]) {
  const f32x16 zero = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int b = 0; b < NB; ++b)
    nacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, an[b]),
                                                      __builtin_bit_cast(bf16x8, ones), zero, 0, 0, 0);
}

// Scores of one tile against all NB blocks of groups and the lane's top-2.
// HOISTED: the |r|^2 parts (norm_terms) were formed once per workgroup and
// start each block's accumulation (four MFMAs per block); else they are the
// block's fifth MFMA, after the four k-steps (an order the error bound allows:
// it holds for any order of the terms).  Block b + 1's MFMAs are interleaved
// with block b's reduction (all in one straight-line region), so the matrix
// cores and the VALU work together.
template <int NB, bool HOISTED>
__device__ __forceinline__ void score_tile(const u32x4 (&af)[NB][4], const u32x4 (&an)[NB], const u32x4& ones,
                                           const f32x16 (&nacc)[NB], const u32x4 (&kf)[4], float& M1, float& M2,
                                           int& B1) {
  const f32x16 zero = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  constexpr int kM = HOISTED ? 4 : 5;  // MFMAs per block
  f32x16 acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    acc[b] = HOISTED ? nacc[b] : zero;
#pragma unroll
    for (int s2 = 0; s2 < 4; ++s2)
      acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, af[b][s2]),
                                                       __builtin_bit_cast(bf16x8, kf[s2]), acc[b], 0, 0, 0);
    if (!HOISTED)
      acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, an[b]),
                                                       __builtin_bit_cast(bf16x8, ones), acc[b], 0, 0, 0);
  }
  M1 = FLT_MAX;
  M2 = FLT_MAX;
  B1 = 0;
#pragma unroll
  for (int b = 0; b < NB; ++b) reduce_block(acc[b], b, M1, M2, B1);
  __builtin_amdgcn_sched_group_barrier(0x008, kM, 0);  // block 0's MFMAs
#pragma unroll
  for (int b = 1; b < NB; ++b)
#pragma unroll
    for (int g = 0; g < kM; ++g) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                  // one MFMA of block b
      __builtin_amdgcn_sched_group_barrier(0x002, HOISTED ? 10 : 8, 0);  // VALU of block b - 1
    }
}
