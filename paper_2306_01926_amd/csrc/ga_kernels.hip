// gfx950 (MI355X) kernels for RITA group attention.
//
// Grouping (Section 4.4): Lloyd K-means on the keys of every (b, h) slice, the
// squared distance expanded as |r|^2 - 2 k.r so that its bulk is the n x N x d
// contraction K R^T.  Aggregation and group softmax: Section 4.2, Eq. 3,
// Algorithm 1.
//
// Kernels, in the order the forward runs them:
//   k_init          C0_j = k_{floor(j n / N)} (or a given init); R = round(C);
//                   canonical fp64 |r_j|^2
//   k_assign_bf16   MFMA 32x32x16 bf16 scores |r_j|^2 - 2 k.r_j with an
//                   in-register top-2 per key; keys whose top-2 gap is inside
//                   a rigorous error band are re-decided with the exact fp64
//                   definition (k_assign_exact's routine)
//   k_assign_exact  fp64 fma-chain scores for every (key, group) (fp32 data)
//   k_bucket        stable counting sort of keys by group (one workgroup per
//                   slice): counts, group offsets, permutation
//   k_segsum        one wave per group sums its members' rows in ascending key
//                   order in fp64 (lane = feature): centroid update or value sums
//   k_attend_prep   bf16 representatives, per-group value means (transposed)
//                   and the log2(count) score bias
//   k_attend_bf16   MFMA scores, block-wise online group softmax, MFMA combine
//   k_attend_f32    the same in fp32 VALU (one thread per query)
#include <hip/hip_runtime.h>

#include <float.h>
#include <math.h>
#include <stdint.h>

#include <mutex>

#include "ga_internal.h"

namespace ga {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kRs = 72;       // LDS row stride (bf16 elements) of the 32x16 MFMA A tiles
constexpr int kAttTpw = 4;    // 32-query tiles per wave in the bf16 attention kernel
constexpr int kAttMaxN = 256; // groups held in LDS by the bf16 attention kernel

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

// Representative of one group row from its fp32 centroid value (lane = feature).
template <class S>
__device__ void finalize_rep(float c, int64_t row, typename S::T* R, double* nrm64, float* nrm32) {
  const int lane = threadIdx.x & 63;
  const float r = S::rep(c);
  S::store(R, row * 64 + lane, r);
  const double nrm = canon_nrm_wave(r);
  if (lane == 0) {
    nrm64[row] = nrm;
    nrm32[row] = (float)nrm;
  }
}

// Exact assignment of one key, cooperatively by a whole wave: lanes take
// groups j = lane, lane + 64, ...; score fma(-2, k.r_j, |r_j|^2) in fp64 with
// the dot product an fma chain over c = 0..63; lowest index among minima.
template <class S>
__device__ int exact_argmin_wave(const typename S::T* __restrict__ krow,
                                 const typename S::T* __restrict__ Rbh,
                                 const double* __restrict__ nrm, int N) {
  const int lane = threadIdx.x & 63;
  double best = INFINITY;
  int bj = 0x7fffffff;
  for (int j = lane; j < N; j += 64) {
    const typename S::T* r = Rbh + (int64_t)j * 64;
    double dot = 0.0;
    for (int c = 0; c < 64; ++c) dot = fma((double)S::load(krow, c), (double)S::load(r, c), dot);
    const double s = fma(-2.0, dot, nrm[j]);
    if (s < best) {
      best = s;
      bj = j;
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const double ob = __shfl_xor(best, off);
    const int oj = __shfl_xor(bj, off);
    if (ob < best || (ob == best && oj < bj)) {
      best = ob;
      bj = oj;
    }
  }
  return bj;
}

// ------------------------------------------------------------------ init
// grid (ceil(N/4), BH), 256 threads: one wave per group, lane = feature.
template <class S>
__global__ __launch_bounds__(256) void k_init(const typename S::T* __restrict__ K,
                                              const float* __restrict__ init, int n, int N,
                                              float* __restrict__ C, typename S::T* __restrict__ R,
                                              double* __restrict__ nrm64, float* __restrict__ nrm32) {
  const int lane = threadIdx.x & 63;
  const int g = __builtin_amdgcn_readfirstlane(blockIdx.x * 4 + (threadIdx.x >> 6));
  const int64_t bh = blockIdx.y;
  if (g >= N) return;
  const int64_t row = bh * N + g;
  const float c = init ? init[row * 64 + lane]
                       : S::load(K, (bh * n + ((int64_t)g * n) / N) * 64 + lane);
  C[row * 64 + lane] = c;
  finalize_rep<S>(c, row, R, nrm64, nrm32);
}

// ------------------------------------------------------------------ assign (bf16, MFMA)
// grid (ceil(tiles / (4 * tpw)), BH), 256 threads.  Each wave owns tpw
// consecutive 32-key tiles.  LDS: -2R as [Npad][kRs] bf16, fl32(|r|^2) [Npad].
//
// MFMA 32x32x16: rows = 32 groups (A = -2R), columns = 32 keys (B = K), the
// accumulator initialised with fl32(|r_j|^2), so each output is the score
// s_ij = |r_j|^2 - 2 k_i.r_j.  Lane l (h = l/32, q = l%32) supplies at k-step s
// features 32h + 8s .. +7 of its row for both operands (the same permutation
// of the contraction axis on both sides), and receives groups
// 8(v/4) + 4h + v%4 of key q in accumulator register v.
//
// Each score is packed with its group index in the low `codebits` mantissa
// bits, so one float min/med3 chain keeps the best and second-best (value and
// index) per key.  If second - best > 2E, where E bounds |packed - exact| (the
// MFMA fp32 accumulation, the fp32 rounding of |r|^2 and the packing), the
// best is provably the exact fp64 argmin; otherwise the key is re-decided by
// exact_argmin_wave.
template <bool FIRST>
__global__ __launch_bounds__(256) void k_assign_bf16(
    const uint16_t* __restrict__ K, const uint16_t* __restrict__ R, const float* __restrict__ nrm32,
    const double* __restrict__ nrm64, float* __restrict__ knorm, int32_t* __restrict__ belong, int n,
    int N, int tpw, float cbound, int codebits) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ double red[4];
  const int Npad = (N + 31) & ~31;
  uint16_t* Rs = (uint16_t*)smem;
  float* n32s = (float*)(smem + (size_t)Npad * kRs * 2);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5, q = lane & 31;
  const int64_t bh = blockIdx.y;
  const uint16_t* Rbh = R + bh * (int64_t)N * 64;

  for (int idx = tid; idx < Npad * 8; idx += 256) {
    const int row = idx >> 3, ch = idx & 7;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (row < N) {
      const u32x4 w = *(const u32x4*)(Rbh + (int64_t)row * 64 + ch * 8);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t lo = __float_as_uint(bf16_to_f32(w[e] & 0xffffu) * -2.0f) >> 16;
        const uint32_t hi = __float_as_uint(bf16_to_f32(w[e] >> 16) * -2.0f) >> 16;
        v[e] = lo | (hi << 16);
      }
    }
    *(u32x4*)(Rs + row * kRs + ch * 8) = v;
  }
  double mx = 0.0;
  for (int j = tid; j < Npad; j += 256) {
    n32s[j] = j < N ? nrm32[bh * N + j] : FLT_MAX;
    if (j < N) mx = fmax(mx, nrm64[bh * N + j]);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mx = fmax(mx, __shfl_xor(mx, off));
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  const double nmax = fmax(fmax(red[0], red[1]), fmax(red[2], red[3]));
  const float nmaxf = (float)nmax * (1.0f + 0x1p-20f);
  const float rmaxf = sqrtf(nmaxf) * (1.0f + 0x1p-20f);

  const int nblk = Npad >> 5;
  const uint32_t keep = ~((1u << codebits) - 1u);
  const uint32_t codemask = (1u << codebits) - 1u;
  uint32_t jc[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) jc[v] = 8 * (v >> 2) + 4 * h + (v & 3);

  const int64_t tile0 = ((int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(wave)) * tpw;
  for (int tt = 0; tt < tpw; ++tt) {
    const int64_t tile = tile0 + tt;
    if (tile * 32 >= n) break;
    const int64_t key = tile * 32 + q;
    const bool valid = key < n;
    const uint16_t* krow = K + (bh * n + (valid ? key : 0)) * 64 + h * 32;
    u32x4 kf[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      kf[s] = u32x4{0u, 0u, 0u, 0u};
      if (valid) kf[s] = *(const u32x4*)(krow + s * 8);
    }
    float kn;
    if (FIRST) {
      float ss = 0.f;
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float lo = bf16_to_f32(kf[s][e] & 0xffffu), hi = bf16_to_f32(kf[s][e] >> 16);
          ss = fmaf(lo, lo, ss);
          ss = fmaf(hi, hi, ss);
        }
      ss += __shfl_xor(ss, 32);
      kn = sqrtf(ss) * (1.0f + 0x1p-16f);
      if (valid && h == 0) knorm[bh * n + key] = kn;
    } else {
      kn = valid ? knorm[bh * n + key] : 0.f;
    }

    float M1 = FLT_MAX, M2 = FLT_MAX;
    for (int blk = 0; blk < nblk; ++blk) {
      f32x16 acc;
      const float* nb = n32s + blk * 32 + 4 * h;
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[v] = nb[8 * (v >> 2) + (v & 3)];
      const uint16_t* ar = Rs + (blk * 32 + q) * kRs + h * 32;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const u32x4 a = *(const u32x4*)(ar + s * 8);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                      __builtin_bit_cast(bf16x8, kf[s]), acc, 0, 0, 0);
      }
      float m1 = FLT_MAX, m2 = FLT_MAX;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float x = __uint_as_float((__float_as_uint(acc[v]) & keep) | jc[v]);
        m2 = __builtin_amdgcn_fmed3f(m1, m2, x);
        m1 = fminf(m1, x);
      }
      const uint32_t bb = (uint32_t)blk << 5;
      m1 = __uint_as_float(__float_as_uint(m1) | bb);
      m2 = __uint_as_float(__float_as_uint(m2) | bb);
      const float nm2 = fminf(fmaxf(M1, m1), fminf(M2, m2));
      M1 = fminf(M1, m1);
      M2 = nm2;
    }
    {
      const float p1 = __shfl_xor(M1, 32), p2 = __shfl_xor(M2, 32);
      const float nm2 = fminf(fmaxf(M1, p1), fminf(M2, p2));
      M1 = fminf(M1, p1);
      M2 = nm2;
    }
    int jstar = (int)(__float_as_uint(M1) & codemask);
    const float E = cbound * (nmaxf + 2.0f * kn * rmaxf) + 1e-30f;
    const bool certain = (M2 > M1 + 2.0f * E) && (jstar < N);
    uint64_t unc = __ballot(valid && !certain && h == 0);
    while (unc) {
      const int b = __ffsll((unsigned long long)unc) - 1;
      unc &= unc - 1;
      const int jb = exact_argmin_wave<BF16>(K + (bh * n + tile * 32 + b) * 64, Rbh, nrm64 + bh * N, N);
      if (q == b) jstar = jb;
    }
    if (valid && h == 0) belong[bh * n + key] = jstar;
  }
}

// ------------------------------------------------------------------ assign (exact)
// grid (ceil(n / (4 * kpw)), BH), 256 threads; each wave decides kpw keys.
template <class S>
__global__ __launch_bounds__(256) void k_assign_exact(const typename S::T* __restrict__ K,
                                                      const typename S::T* __restrict__ R,
                                                      const double* __restrict__ nrm64,
                                                      int32_t* __restrict__ belong, int n, int N,
                                                      int kpw) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t bh = blockIdx.y;
  const int64_t key0 = ((int64_t)blockIdx.x * 4 + wave) * kpw;
  for (int k = 0; k < kpw; ++k) {
    const int64_t key = key0 + k;
    if (key >= n) break;
    const int jb = exact_argmin_wave<S>(K + (bh * n + key) * 64, R + bh * (int64_t)N * 64,
                                        nrm64 + bh * N, N);
    if (lane == 0) belong[bh * n + key] = jb;
  }
}

// ------------------------------------------------------------------ bucket
__device__ __forceinline__ int wave_incl_scan(int x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int t = __shfl_up(x, d);
    if (lane >= d) x += t;
  }
  return x;
}

// Stable counting sort of one slice's keys by group; grid BH, 1024 threads.
// LDS: per-wave 64-bit lane masks [16][N], counts [N], running offsets [N].
// Within a 1024-key chunk, a key's rank among same-group keys is the number
// of lower lanes in its wave with the same group (popcount of the OR-ed lane
// mask) plus the members of that group in the lower waves of the chunk.
__global__ __launch_bounds__(1024) void k_bucket(const int32_t* __restrict__ belong, int n, int N,
                                                 int32_t* __restrict__ perm, int32_t* __restrict__ goff,
                                                 int32_t* __restrict__ count) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int wsum[16];
  unsigned long long* wmask = (unsigned long long*)smem;
  int32_t* cnt = (int32_t*)(wmask + 16 * N);
  int32_t* run = cnt + N;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t bh = blockIdx.x;
  const int32_t* a = belong + bh * n;

  for (int g = tid; g < N; g += 1024) cnt[g] = 0;
  for (int x = tid; x < 16 * N; x += 1024) wmask[x] = 0ull;
  __syncthreads();
  for (int i = tid; i < n; i += 1024) {
    const int g = a[i];
    if ((unsigned)g < (unsigned)N) atomicAdd(&cnt[g], 1);
  }
  __syncthreads();
  const int v = tid < N ? cnt[tid] : 0;
  const int incl = wave_incl_scan(v);
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    const int t = lane < 16 ? wsum[lane] : 0;
    const int ti = wave_incl_scan(t);
    if (lane < 16) wsum[lane] = ti - t;
  }
  __syncthreads();
  if (tid < N) {
    const int ex = incl - v + wsum[wave];
    run[tid] = ex;
    goff[bh * N + tid] = ex;
    count[bh * N + tid] = v;
  }
  __syncthreads();

  const unsigned long long below = (1ull << lane) - 1ull;
  for (int base = 0; base < n; base += 1024) {
    const int i = base + tid;
    const int g = i < n ? a[i] : -1;
    const bool ok = (unsigned)g < (unsigned)N;
    if (ok) atomicOr(&wmask[wave * N + g], 1ull << lane);
    __syncthreads();
    unsigned long long m = 0ull;
    int rank = 0;
    if (ok) {
      m = wmask[wave * N + g];
      rank = __popcll(m & below);
      int pre = 0;
      for (int w2 = 0; w2 < wave; ++w2) pre += __popcll(wmask[w2 * N + g]);
      perm[bh * n + run[g] + pre + rank] = i;
    }
    __syncthreads();
    if (ok && rank == 0) {
      atomicAdd(&run[g], __popcll(m));
      wmask[wave * N + g] = 0ull;
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------ segmented sums
// grid (ceil(N/4), BH), 256 threads: one wave per group, lane = feature.  The
// group's members are perm[goff .. goff + count) in ascending key order and
// are summed in that order in fp64.  UPDATE: centroid = (float)(sum / count)
// (an empty group keeps its centroid) and its representative; otherwise the
// fp32 rounding of the value sum.
template <class S, bool UPDATE>
__global__ __launch_bounds__(256) void k_segsum(const typename S::T* __restrict__ X,
                                                const int32_t* __restrict__ perm,
                                                const int32_t* __restrict__ goff,
                                                const int32_t* __restrict__ count, int n, int N,
                                                float* __restrict__ out, typename S::T* __restrict__ R,
                                                double* __restrict__ nrm64, float* __restrict__ nrm32) {
  const int lane = threadIdx.x & 63;
  const int g = __builtin_amdgcn_readfirstlane(blockIdx.x * 4 + (threadIdx.x >> 6));
  const int64_t bh = blockIdx.y;
  if (g >= N) return;
  const int64_t row = bh * N + g;
  const int st = goff[row], cnt = count[row];
  const int32_t* P = perm + bh * n + st;
  const typename S::T* Xb = X + bh * (int64_t)n * 64 + lane;
  double acc = 0.0;
  int x = 0;
  for (; x + 4 <= cnt; x += 4) {
    const int i0 = P[x], i1 = P[x + 1], i2 = P[x + 2], i3 = P[x + 3];
    const float v0 = S::load(Xb, (int64_t)i0 * 64), v1 = S::load(Xb, (int64_t)i1 * 64);
    const float v2 = S::load(Xb, (int64_t)i2 * 64), v3 = S::load(Xb, (int64_t)i3 * 64);
    acc += (double)v0;
    acc += (double)v1;
    acc += (double)v2;
    acc += (double)v3;
  }
  for (; x < cnt; ++x) acc += (double)S::load(Xb, (int64_t)P[x] * 64);
  if (UPDATE) {
    float c;
    if (cnt > 0) {
      c = (float)(acc / (double)cnt);
      out[row * 64 + lane] = c;
    } else {
      c = out[row * 64 + lane];
    }
    finalize_rep<S>(c, row, R, nrm64, nrm32);
  } else {
    out[row * 64 + lane] = (float)acc;
  }
}

// ------------------------------------------------------------------ attention (bf16)
// grid (ceil(Npad/4), BH), 256 threads: one wave per (padded) group, lane = feature.
// Vt holds the group's value MEAN vsum_j / count_j (bf16) so that the count
// weight can move into the exponent: o_i = sum_j c_j e_ij mu_j / sum_j c_j e_ij
// with c_j e_ij = exp2(t_ij + log2 c_j).  ginit_j = log2(c_j) / sl2e is added to
// the score accumulator (-inf for an empty group, which drops it).
__global__ __launch_bounds__(256) void k_attend_prep(const float* __restrict__ centroid,
                                                     const int32_t* __restrict__ count,
                                                     const float* __restrict__ vsum, float inv_sl2e,
                                                     int N, int vts, uint16_t* __restrict__ Rq,
                                                     uint16_t* __restrict__ Vt, float* __restrict__ ginit) {
  const int lane = threadIdx.x & 63;
  const int g = __builtin_amdgcn_readfirstlane(blockIdx.x * 4 + (threadIdx.x >> 6));
  const int64_t bh = blockIdx.y;
  const int Npad = (N + 31) & ~31;
  if (g >= Npad) return;
  const bool valid = g < N;
  const int64_t row = bh * N + g;
  const int cnt = valid ? count[row] : 0;
  if (Rq && valid) Rq[row * 64 + lane] = (uint16_t)f32_to_bf16(centroid[row * 64 + lane]);
  const float mu = cnt > 0 ? vsum[row * 64 + lane] / (float)cnt : 0.f;
  Vt[(bh * 64 + lane) * vts + g] = (uint16_t)f32_to_bf16(mu);
  if (lane == 0) ginit[bh * Npad + g] = cnt > 0 ? log2f((float)cnt) * inv_sl2e : -INFINITY;
}

// grid (ceil(tiles / (4 * kAttTpw)), BH), 256 threads, N <= kAttMaxN.
// LDS: sign(scale) R as [Npad][kRs] bf16, Vt as [64][vts] bf16, ginit [Npad].
// Scores: MFMA with A = R rows (32 groups), B = Q tile (32 queries); accumulator
// init ginit.  t = acc * sl2e; online max per 32-group block, rescaled only when
// the block max exceeds the running max by more than 8 (log2 units).  Combine:
// MFMA with A = Vt rows (32 features x 16 groups), B = bf16(exp2(t - m)) taken
// straight from the score registers (the group order of the contraction axis
// is the score layout's, applied identically to A).
__global__ __launch_bounds__(256) void k_attend_bf16(const uint16_t* __restrict__ Q,
                                                     const uint16_t* __restrict__ R,
                                                     const uint16_t* __restrict__ Vt,
                                                     const float* __restrict__ ginit, int n, int N,
                                                     int vts, float sl2e, uint32_t rsign,
                                                     uint16_t* __restrict__ O) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int Npad = (N + 31) & ~31;
  uint16_t* Rs = (uint16_t*)smem;
  uint16_t* Vs = Rs + Npad * kRs;
  float* gi = (float*)(Vs + 64 * vts);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5, q = lane & 31;
  const int64_t bh = blockIdx.y;
  const uint16_t* Rbh = R + bh * (int64_t)N * 64;
  for (int idx = tid; idx < Npad * 8; idx += 256) {
    const int row = idx >> 3, ch = idx & 7;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (row < N) {
      v = *(const u32x4*)(Rbh + (int64_t)row * 64 + ch * 8);
      v ^= u32x4{rsign, rsign, rsign, rsign};
    }
    *(u32x4*)(Rs + row * kRs + ch * 8) = v;
  }
  const uint16_t* Vbh = Vt + bh * 64 * (int64_t)vts;
  // rows of Vt are 8-byte aligned (vts = 128k + 4 keeps the combine's LDS reads conflict-free)
  for (int idx = tid; idx < 64 * (Npad / 4); idx += 256) {
    const int row = idx / (Npad / 4), ch = idx % (Npad / 4);
    *(u32x2*)(Vs + row * vts + ch * 4) = *(const u32x2*)(Vbh + (int64_t)row * vts + ch * 4);
  }
  bool nonempty = false;
  for (int j = tid; j < Npad; j += 256) {
    const float x = ginit[bh * Npad + j];
    gi[j] = x;
    nonempty |= (x != -INFINITY);
  }
  const int any = __syncthreads_or(nonempty);
  const int nblk = Npad >> 5;

  const int64_t tile0 = ((int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(wave)) * kAttTpw;
  for (int tt = 0; tt < kAttTpw; ++tt) {
    const int64_t tile = tile0 + tt;
    if (tile * 32 >= n) break;
    const int64_t qi = tile * 32 + q;
    const bool valid = qi < n;
    uint16_t* orow = O + (bh * n + (valid ? qi : 0)) * 64;
    if (!any) {
      if (valid)
        for (int c = h * 32; c < h * 32 + 32; c += 8) *(u32x4*)(orow + c) = u32x4{0u, 0u, 0u, 0u};
      continue;
    }
    const uint16_t* qrow = Q + (bh * n + (valid ? qi : 0)) * 64 + h * 32;
    u32x4 qf[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      qf[s] = u32x4{0u, 0u, 0u, 0u};
      if (valid) qf[s] = *(const u32x4*)(qrow + s * 8);
    }
    f32x16 o0, o1;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      o0[v] = 0.f;
      o1[v] = 0.f;
    }
    float mt = -INFINITY, ssum = 0.f;
    for (int blk = 0; blk < nblk; ++blk) {
      f32x16 acc;
      const float* gb = gi + blk * 32 + 4 * h;
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[v] = gb[8 * (v >> 2) + (v & 3)];
      const uint16_t* ar = Rs + (blk * 32 + q) * kRs + h * 32;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const u32x4 a = *(const u32x4*)(ar + s * 8);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                      __builtin_bit_cast(bf16x8, qf[s]), acc, 0, 0, 0);
      }
      float bm = acc[0];
#pragma unroll
      for (int v = 1; v < 16; ++v) bm = fmaxf(bm, acc[v]);
      bm = fmaxf(bm, __shfl_xor(bm, 32));
      if (bm == -INFINITY) continue;  // every group of this block is empty (uniform)
      const float bmt = bm * sl2e;
      if (bmt > mt + 8.0f) {
        const float alpha = exp2f(mt - bmt);
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          o0[v] *= alpha;
          o1[v] *= alpha;
        }
        ssum *= alpha;
        mt = bmt;
      }
      float e[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        e[v] = exp2f(fmaf(acc[v], sl2e, -mt));
        ssum += e[v];
      }
      u32x4 b0, b1;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        b0[w] = pack_bf16x2(e[2 * w], e[2 * w + 1]);
        b1[w] = pack_bf16x2(e[8 + 2 * w], e[8 + 2 * w + 1]);
      }
#pragma unroll
      for (int sp = 0; sp < 2; ++sp) {
        const int gcol = blk * 32 + 16 * sp + 4 * h;
        const u32x4 bsp = sp == 0 ? b0 : b1;
        {
          const uint16_t* vr = Vs + q * vts + gcol;
          const u32x2 lo = *(const u32x2*)vr, hi = *(const u32x2*)(vr + 8);
          const u32x4 a = {lo[0], lo[1], hi[0], hi[1]};
          o0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, bsp), o0, 0, 0, 0);
        }
        {
          const uint16_t* vr = Vs + (32 + q) * vts + gcol;
          const u32x2 lo = *(const u32x2*)vr, hi = *(const u32x2*)(vr + 8);
          const u32x4 a = {lo[0], lo[1], hi[0], hi[1]};
          o1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, bsp), o1, 0, 0, 0);
        }
      }
    }
    const float stot = ssum + __shfl_xor(ssum, 32);
    const float inv = 1.0f / stot;
    if (valid) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        u32x2 w0 = {pack_bf16x2(o0[4 * r] * inv, o0[4 * r + 1] * inv),
                    pack_bf16x2(o0[4 * r + 2] * inv, o0[4 * r + 3] * inv)};
        u32x2 w1 = {pack_bf16x2(o1[4 * r] * inv, o1[4 * r + 1] * inv),
                    pack_bf16x2(o1[4 * r + 2] * inv, o1[4 * r + 3] * inv)};
        *(u32x2*)(orow + 8 * r + 4 * h) = w0;
        *(u32x2*)(orow + 32 + 8 * r + 4 * h) = w1;
      }
    }
  }
}

// ------------------------------------------------------------------ attention (fp32)
// grid (ceil(n/256), BH), 256 threads, one query per thread; groups stream
// through LDS in chunks of 64 (centroid rows and value sums, fp32).  Online
// softmax with the exact running max over non-empty groups.
__global__ __launch_bounds__(256) void k_attend_f32(const float* __restrict__ Q,
                                                    const float* __restrict__ centroid,
                                                    const int32_t* __restrict__ count,
                                                    const float* __restrict__ vsum, int n, int N,
                                                    float scale, float* __restrict__ O) {
  __shared__ float Rs[64][65];
  __shared__ float Vs[64][65];
  __shared__ int cs[64];
  const int tid = threadIdx.x;
  const int64_t bh = blockIdx.y;
  const int64_t qi = (int64_t)blockIdx.x * 256 + tid;
  const bool valid = qi < n;
  float qv[64], o[64];
  const float* qrow = Q + (bh * n + (valid ? qi : 0)) * 64;
#pragma unroll
  for (int c = 0; c < 64; ++c) {
    qv[c] = valid ? qrow[c] : 0.f;
    o[c] = 0.f;
  }
  float m = -INFINITY, ssum = 0.f;
  for (int base = 0; base < N; base += 64) {
    __syncthreads();
    for (int x = tid; x < 64 * 64; x += 256) {
      const int j = x >> 6, c = x & 63;
      const bool in = base + j < N;
      Rs[j][c] = in ? centroid[(bh * N + base + j) * 64 + c] : 0.f;
      Vs[j][c] = in ? vsum[(bh * N + base + j) * 64 + c] : 0.f;
    }
    if (tid < 64) cs[tid] = base + tid < N ? count[bh * N + base + tid] : 0;
    __syncthreads();
    const int lim = min(64, N - base);
    for (int j = 0; j < lim; ++j) {
      const int cj = cs[j];
      if (cj <= 0) continue;
      float dot = 0.f;
#pragma unroll
      for (int c = 0; c < 64; ++c) dot = fmaf(qv[c], Rs[j][c], dot);
      const float p = scale * dot;
      if (p > m) {
        const float alpha = expf(m - p);
#pragma unroll
        for (int c = 0; c < 64; ++c) o[c] *= alpha;
        ssum *= alpha;
        m = p;
      }
      const float e = expf(p - m);
      ssum = fmaf((float)cj, e, ssum);
#pragma unroll
      for (int c = 0; c < 64; ++c) o[c] = fmaf(e, Vs[j][c], o[c]);
    }
  }
  if (valid) {
    const float inv = ssum > 0.f ? 1.0f / ssum : 0.f;
    float* orow = O + (bh * n + qi) * 64;
#pragma unroll
    for (int c = 0; c < 64; ++c) orow[c] = o[c] * inv;
  }
}

size_t assign_lds(int N) {
  const int Npad = (N + 31) & ~31;
  return (size_t)Npad * kRs * 2 + (size_t)Npad * 4;
}
size_t bucket_lds(int N) { return (size_t)16 * N * 8 + (size_t)2 * N * 4; }
size_t attend_lds(int N) {
  const int Npad = (N + 31) & ~31;
  return (size_t)Npad * kRs * 2 + (size_t)64 * vt_stride(N) * 2 + (size_t)Npad * 4;
}

// Raise the dynamic-LDS limit of the kernels that can exceed 64 KB to the
// most they ever request.  A failure here is not fatal (the launch reports any
// real problem), so the error it leaves behind is cleared.
void set_lds_limits() {
  static std::once_flag once;
  std::call_once(once, [] {
    (void)hipFuncSetAttribute((const void*)k_assign_bf16<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)assign_lds(kMaxGroups));
    (void)hipFuncSetAttribute((const void*)k_assign_bf16<false>, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)assign_lds(kMaxGroups));
    (void)hipFuncSetAttribute((const void*)k_bucket, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)bucket_lds(kMaxGroups));
    (void)hipFuncSetAttribute((const void*)k_attend_bf16, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)attend_lds(kAttMaxN));
    (void)hipGetLastError();
  });
}

inline unsigned cdiv(int64_t a, int64_t b) { return (unsigned)((a + b - 1) / b); }

}  // namespace

int vt_stride(int N) {
  const int Npad = (N + 31) & ~31;
  return ((Npad + 127) / 128) * 128 + 4;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t workspace_layout(const Dims& d, Workspace* ws, void* base) {
  const int64_t BH = d.BH, n = d.n, N = d.N;
  const int64_t Npad = (N + 31) & ~31;
  const size_t es = d.dtype == 1 ? 2 : 4;
  size_t off = 0;
  char* b = (char*)base;
  auto take = [&](size_t bytes) -> void* {
    void* p = b ? (void*)(b + off) : nullptr;
    off += align256(bytes);
    return p;
  };
  Workspace w{};
  w.C = (float*)take(BH * N * 64 * 4);
  w.R = take(BH * N * 64 * es);
  w.nrm64 = (double*)take(BH * N * 8);
  w.nrm32 = (float*)take(BH * N * 4);
  w.knorm = (float*)take(BH * n * 4);
  w.belong = (int32_t*)take(BH * n * 4);
  w.perm = (int32_t*)take(BH * n * 4);
  w.goff = (int32_t*)take(BH * N * 4);
  w.count = (int32_t*)take(BH * N * 4);
  w.vsum = (float*)take(BH * N * 64 * 4);
  w.Rq = (uint16_t*)take(BH * N * 64 * 2);
  w.Vt = (uint16_t*)take(BH * 64 * (int64_t)vt_stride((int)N) * 2);
  w.ginit = (float*)take(BH * Npad * 4);
  if (ws) *ws = w;
  return off;
}

hipError_t launch_init(const Dims& d, const void* K, const float* init, float* C, void* R,
                       double* nrm64, float* nrm32, hipStream_t st) {
  TimedLaunch timed("init", st);
  const dim3 grid(cdiv(d.N, 4), (unsigned)d.BH), block(256);
  if (d.dtype == 1)
    hipLaunchKernelGGL(k_init<BF16>, grid, block, 0, st, (const uint16_t*)K, init, d.n, d.N, C,
                       (uint16_t*)R, nrm64, nrm32);
  else
    hipLaunchKernelGGL(k_init<F32>, grid, block, 0, st, (const float*)K, init, d.n, d.N, C, (float*)R,
                       nrm64, nrm32);
  return hipGetLastError();
}

hipError_t launch_assign(const Dims& d, const void* K, const void* R, const float* nrm32,
                         const double* nrm64, float* knorm, int32_t* belong, bool first,
                         hipStream_t st) {
  TimedLaunch timed("assign", st);
  set_lds_limits();
  if (d.dtype == 1) {
    const int64_t tiles = (d.n + 31) / 32;
    int64_t tpw = (d.BH * tiles) / (4 * 2048);
    tpw = tpw < 1 ? 1 : (tpw > 8 ? 8 : tpw);
    const int Npad = (d.N + 31) & ~31;
    int codebits = 5;
    while ((1 << codebits) < Npad) ++codebits;
    // |MFMA fp32 accumulation error| <= (d + 4) 2^-24 * 2 * sum|terms| (each of the
    // d products and the init rounded at most once, sequential model, 2x margin);
    // packing the index moves a value by < 2^(codebits - 23) of its magnitude.
    const float cbound = ((float)(kD + 4) * 0x1p-23f + ldexpf(1.0f, codebits - 23)) * (1.0f + 0x1p-10f);
    const dim3 grid(cdiv(tiles, 4 * tpw), (unsigned)d.BH), block(256);
    const size_t lds = assign_lds(d.N);
    if (first)
      hipLaunchKernelGGL(k_assign_bf16<true>, grid, block, lds, st, (const uint16_t*)K, (const uint16_t*)R,
                         nrm32, nrm64, knorm, belong, d.n, d.N, (int)tpw, cbound, codebits);
    else
      hipLaunchKernelGGL(k_assign_bf16<false>, grid, block, lds, st, (const uint16_t*)K, (const uint16_t*)R,
                         nrm32, nrm64, knorm, belong, d.n, d.N, (int)tpw, cbound, codebits);
  } else {
    const int kpw = 4;
    const dim3 grid(cdiv(d.n, 4 * kpw), (unsigned)d.BH), block(256);
    hipLaunchKernelGGL(k_assign_exact<F32>, grid, block, 0, st, (const float*)K, (const float*)R, nrm64,
                       belong, d.n, d.N, kpw);
  }
  return hipGetLastError();
}

hipError_t launch_bucket(const Dims& d, const int32_t* belong, int32_t* perm, int32_t* goff,
                         int32_t* count, hipStream_t st) {
  TimedLaunch timed("bucket", st);
  set_lds_limits();
  hipLaunchKernelGGL(k_bucket, dim3((unsigned)d.BH), dim3(1024), bucket_lds(d.N), st, belong, d.n, d.N,
                     perm, goff, count);
  return hipGetLastError();
}

hipError_t launch_update(const Dims& d, const void* K, const int32_t* perm, const int32_t* goff,
                         const int32_t* count, float* C, void* R, double* nrm64, float* nrm32,
                         hipStream_t st) {
  TimedLaunch timed("update", st);
  const dim3 grid(cdiv(d.N, 4), (unsigned)d.BH), block(256);
  if (d.dtype == 1)
    hipLaunchKernelGGL((k_segsum<BF16, true>), grid, block, 0, st, (const uint16_t*)K, perm, goff, count,
                       d.n, d.N, C, (uint16_t*)R, nrm64, nrm32);
  else
    hipLaunchKernelGGL((k_segsum<F32, true>), grid, block, 0, st, (const float*)K, perm, goff, count, d.n,
                       d.N, C, (float*)R, nrm64, nrm32);
  return hipGetLastError();
}

hipError_t launch_valuesum(const Dims& d, const void* V, const int32_t* perm, const int32_t* goff,
                           const int32_t* count, float* vsum, hipStream_t st) {
  TimedLaunch timed("valuesum", st);
  const dim3 grid(cdiv(d.N, 4), (unsigned)d.BH), block(256);
  if (d.dtype == 1)
    hipLaunchKernelGGL((k_segsum<BF16, false>), grid, block, 0, st, (const uint16_t*)V, perm, goff, count,
                       d.n, d.N, vsum, (uint16_t*)nullptr, (double*)nullptr, (float*)nullptr);
  else
    hipLaunchKernelGGL((k_segsum<F32, false>), grid, block, 0, st, (const float*)V, perm, goff, count, d.n,
                       d.N, vsum, (float*)nullptr, (double*)nullptr, (float*)nullptr);
  return hipGetLastError();
}

static float clamp_sl2e(float scale) {
  const float s = fabsf(scale) * 1.4426950408889634f;
  return s < 1e-30f ? 1e-30f : s;
}

hipError_t launch_attend_prep(const Dims& d, const float* centroid, const int32_t* count,
                              const float* vsum, float scale, uint16_t* Rq, uint16_t* Vt, float* ginit,
                              bool make_rq, hipStream_t st) {
  TimedLaunch timed("attend_prep", st);
  const int Npad = (d.N + 31) & ~31;
  const dim3 grid(cdiv(Npad, 4), (unsigned)d.BH), block(256);
  hipLaunchKernelGGL(k_attend_prep, grid, block, 0, st, centroid, count, vsum, 1.0f / clamp_sl2e(scale), d.N,
                     vt_stride(d.N), make_rq ? Rq : (uint16_t*)nullptr, Vt, ginit);
  return hipGetLastError();
}

hipError_t launch_attend(const Dims& d, const void* Q, const void* R, const uint16_t* Vt,
                         const float* ginit, const float* centroid, const int32_t* count,
                         const float* vsum, float scale, void* O, hipStream_t st) {
  TimedLaunch timed("attend", st);
  set_lds_limits();
  if (d.dtype == 1) {
    if (d.N > kAttMaxN) return hipErrorInvalidValue;
    const int64_t tiles = (d.n + 31) / 32;
    const dim3 grid(cdiv(tiles, 4 * kAttTpw), (unsigned)d.BH), block(256);
    const uint32_t rsign = scale < 0.f ? 0x80008000u : 0u;
    hipLaunchKernelGGL(k_attend_bf16, grid, block, attend_lds(d.N), st, (const uint16_t*)Q,
                       (const uint16_t*)R, Vt, ginit, d.n, d.N, vt_stride(d.N), clamp_sl2e(scale), rsign,
                       (uint16_t*)O);
  } else {
    const dim3 grid(cdiv(d.n, 256), (unsigned)d.BH), block(256);
    hipLaunchKernelGGL(k_attend_f32, grid, block, 0, st, (const float*)Q, centroid, count, vsum, d.n, d.N,
                       scale, (float*)O);
  }
  return hipGetLastError();
}

}  // namespace ga
