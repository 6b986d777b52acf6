// gfx950 (MI355X) merge plan of the adaptive group count (Section 5.1).
//
// RITA lowers the group count N during training by merging groups whose merge
// keeps the attention error bound eps:
//   - Lemma 1: if every key lies within dthr of its group's representative
//     and dthr <= ln(eps) / (2 R'), every restored attention weight is within
//     a factor eps of the exact one; R' bounds the scaled query norms, which is
//     what the proof uses: R' = |scale| max_i |q_i|.
//   - Lemma 2 and the simplified rule of Eq. 5: with the groups halved into
//     S1 = [0, ceil(N/2)) and S2 = [ceil(N/2), N), a group j of S2 can merge
//     into a group i of S1 when |c_i - c_j| + rad_i <= dthr and
//     |c_j - c_i| + rad_j <= dthr / 2 (rad_g: largest member distance to the
//     centroid c_g); the S2 groups marked this way are the D groups that go.
//
// k_merge_zero, k_merge_norms, k_merge_pairs: the slice's fp32 centroids go to
// LDS (row stride 65 floats: lanes reading different groups' rows at the same
// feature hit different banks); one pass over the queries and keys, split
// over up to 16 workgroups per slice, computes the largest squared query norm
// and, per group, the largest squared member distance (64-bit max on the bit
// patterns of the non-negative doubles, in LDS and then in global memory:
// order-free, so the result does not depend on the schedule); then one
// workgroup per slice tests every (i in S1, j in S2) pair and an LDS minimum
// keeps the lowest partner of each j.
//
// Every decision is taken in fp64 with the operations of the definition:
// differences formed exactly, squares summed as fma chains over the features
// 0..63 from 0, IEEE square roots, dthr = log_eps / (2 (|scale| qmax)), so the
// marks are bit-for-bit those of the fp64 CPU definition.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "ga_internal.h"

#pragma clang fp contract(off)

namespace ga {
namespace {

constexpr int kMergeThreads = 512;
constexpr int kMergeMaxN = 256;
constexpr int kCs = 65;  // LDS row stride (floats) of the centroids

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// The slice's N x 64 fp32 centroids to LDS (row stride kCs), eight loads per
// thread issued (index clamped) before any of them is stored.
__device__ __forceinline__ void stage_centroids(const float* __restrict__ cen, int N, float* cs) {
  const int tid = threadIdx.x, total = N * 64;
  for (int base = 0; base < total; base += 8 * kMergeThreads) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = cen[min(base + tid + u * kMergeThreads, total - 1)];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int x = base + tid + u * kMergeThreads;
      if (x < total) cs[(x >> 6) * kCs + (x & 63)] = v[u];
    }
  }
}

// Raw rows (loaded as 16-byte vectors) and their exact fp64 elements.
struct F32In {
  typedef float T;
  static constexpr int kVec = 16;  // 16-byte vectors per 64-feature row
  __device__ static void load(const float* p, u32x4 (&v)[16]) {
#pragma unroll
    for (int u = 0; u < 16; ++u) v[u] = *(const u32x4*)(p + 4 * u);
  }
  __device__ static double at(const u32x4 (&v)[16], int c) { return (double)__uint_as_float(v[c >> 2][c & 3]); }
};

struct BF16In {
  typedef uint16_t T;
  static constexpr int kVec = 8;
  __device__ static void load(const uint16_t* p, u32x4 (&v)[8]) {
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = *(const u32x4*)(p + 8 * u);
  }
  __device__ static double at(const u32x4 (&v)[8], int c) {
    const uint32_t w = v[c >> 3][(c >> 1) & 3];
    return (double)__uint_as_float((c & 1) ? (w & 0xffff0000u) : (w << 16));
  }
};

// Squared distance maxima.  grid (parts, BH), 512 threads: workgroup x of a
// slice takes keys [x n / parts, (x + 1) n / parts).  The largest squared
// member distance of each group goes to rad2[bh][g] and the largest squared
// query norm to qmax2[bh], both as bit patterns of non-negative doubles
// combined with 64-bit max (order-free); both start at 0 (k_merge_zero).
template <class S>
__global__ __launch_bounds__(kMergeThreads) void k_merge_norms(
    const typename S::T* __restrict__ Q, const typename S::T* __restrict__ K, const int32_t* __restrict__ belong,
    const float* __restrict__ centroid, int n, int N, unsigned long long* __restrict__ rad2g,
    unsigned long long* __restrict__ qmax2g) {
  __shared__ float cs[kMergeMaxN * kCs];
  __shared__ unsigned long long rad2[kMergeMaxN];
  __shared__ double wmax[kMergeThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t bh = blockIdx.y;
  const int i0 = (int)((int64_t)blockIdx.x * n / gridDim.x), i1 = (int)((int64_t)(blockIdx.x + 1) * n / gridDim.x);
  stage_centroids(centroid + bh * N * 64, N, cs);
  for (int g = tid; g < N; g += kMergeThreads) rad2[g] = 0ull;  // bits of +0.0
  __syncthreads();
  double qmax2 = 0.0;
  // per key: its query row, group and key row are requested together (the
  // key row's address does not depend on the group), then the two chains run
  for (int i = i0 + tid; i < i1; i += kMergeThreads) {
    u32x4 qv[S::kVec], kv[S::kVec];
    S::load(Q + (bh * n + i) * 64, qv);
    const int g = belong[bh * n + i];
    S::load(K + (bh * n + i) * 64, kv);
    double acc = 0.0;
#pragma unroll
    for (int c = 0; c < 64; ++c) {
      const double xq = S::at(qv, c);
      acc = __builtin_fma(xq, xq, acc);
    }
    qmax2 = acc > qmax2 ? acc : qmax2;
    if ((unsigned)g >= (unsigned)N) continue;
    double r2 = 0.0;
#pragma unroll
    for (int c = 0; c < 64; ++c) {
      const double t = S::at(kv, c) - (double)cs[g * kCs + c];
      r2 = __builtin_fma(t, t, r2);
    }
    atomicMax(&rad2[g], (unsigned long long)__double_as_longlong(r2));
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const double o = __shfl_xor(qmax2, off);
    qmax2 = o > qmax2 ? o : qmax2;
  }
  if (lane == 0) wmax[wave] = qmax2;
  __syncthreads();
  for (int g = tid; g < N; g += kMergeThreads)
    if (rad2[g]) atomicMax(&rad2g[bh * N + g], rad2[g]);
  if (tid == 0) {
    double m = wmax[0];
#pragma unroll
    for (int w = 1; w < kMergeThreads / 64; ++w) m = wmax[w] > m ? wmax[w] : m;
    atomicMax(&qmax2g[bh], (unsigned long long)__double_as_longlong(m));
  }
}

// grid (ceil(BH (N + 1) / 256)), 256 threads: zero the maxima.
__global__ __launch_bounds__(256) void k_merge_zero(unsigned long long* __restrict__ rad2g,
                                                    unsigned long long* __restrict__ qmax2g, int64_t BH, int N) {
  const int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (x < BH * N) rad2g[x] = 0ull;
  else if (x < BH * N + BH) qmax2g[x - BH * N] = 0ull;
}

// grid (BH), 512 threads: the threshold and Eq. 5 on every (i in S1, j in S2)
// pair of non-empty groups; rad2g / qmax2g (the bits in radius / dthr) are
// replaced by the radii and the threshold.
__global__ __launch_bounds__(kMergeThreads) void k_merge_pairs(
    const float* __restrict__ centroid, const int32_t* __restrict__ count, int N, double abs_scale, double log_eps,
    double* __restrict__ radius, double* __restrict__ dthr, int32_t* __restrict__ partner,
    int32_t* __restrict__ merges) {
  __shared__ float cs[kMergeMaxN * kCs];
  __shared__ double rad[kMergeMaxN];
  __shared__ int cnt[kMergeMaxN], best[kMergeMaxN];
  __shared__ int nmarked;
  const int tid = threadIdx.x;
  const int64_t bh = blockIdx.x;
  stage_centroids(centroid + bh * N * 64, N, cs);
  for (int g = tid; g < N; g += kMergeThreads) {
    rad[g] = __builtin_sqrt(radius[bh * N + g]);  // radius holds the squared maximum here
    cnt[g] = count[bh * N + g];
    best[g] = 0x7fffffff;
  }
  if (tid == 0) nmarked = 0;
  const double t = log_eps / (2.0 * (abs_scale * __builtin_sqrt(dthr[bh])));
  const double t2 = 0.5 * t;
  __syncthreads();
  const int half = (N + 1) / 2, nj = N - half;
  for (int p = tid; p < half * nj; p += kMergeThreads) {
    const int i = p % half, j = half + p / half;
    if (cnt[i] <= 0 || cnt[j] <= 0) continue;
    double d2 = 0.0;
#pragma unroll 16
    for (int c = 0; c < 64; ++c) {
      const double u = (double)cs[i * kCs + c] - (double)cs[j * kCs + c];
      d2 = __builtin_fma(u, u, d2);
    }
    const double dij = __builtin_sqrt(d2);
    if (dij + rad[i] <= t && dij + rad[j] <= t2) atomicMin(&best[j], i);
  }
  __syncthreads();
  for (int g = tid; g < N; g += kMergeThreads) {
    radius[bh * N + g] = rad[g];
    const int pj = g >= half && best[g] != 0x7fffffff ? best[g] : -1;
    partner[bh * N + g] = pj;
    if (pj >= 0) atomicAdd(&nmarked, 1);
  }
  __syncthreads();
  if (tid == 0) {
    merges[bh] = nmarked;
    dthr[bh] = t;
  }
}

}  // namespace

int merge_max_groups() { return kMergeMaxN; }

hipError_t launch_merge_plan(const Dims& d, const void* Q, const void* K, const int32_t* belong,
                             const float* centroid, const int32_t* count, double abs_scale, double log_eps,
                             double* radius, double* dthr, int32_t* partner, int32_t* merges, hipStream_t st) {
  // the squared maxima are accumulated as bits in the radius and dthr outputs
  unsigned long long* rad2g = (unsigned long long*)radius;
  unsigned long long* qmax2g = (unsigned long long*)dthr;
  {
    TimedLaunch tl("merge_zero", st);
    const int64_t total = d.BH * (d.N + 1);
    hipLaunchKernelGGL(k_merge_zero, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, rad2g, qmax2g, d.BH,
                       d.N);
  }
  // at least about 1000 keys per workgroup, at most 16 workgroups per slice,
  // and no more than one round of about 512 workgroups (two per CU) in all:
  // every workgroup stages the slice's centroids
  const int64_t round_parts = (512 + d.BH - 1) / d.BH;
  int parts = d.n < 1000 ? 1 : (d.n / 1000 > 16 ? 16 : d.n / 1000);
  if (parts > round_parts) parts = (int)round_parts;
  {
    TimedLaunch tl("merge_norms", st);
    if (d.dtype == 1)
      hipLaunchKernelGGL(k_merge_norms<BF16In>, dim3(parts, (unsigned)d.BH), dim3(kMergeThreads), 0, st,
                         (const uint16_t*)Q, (const uint16_t*)K, belong, centroid, d.n, d.N, rad2g, qmax2g);
    else
      hipLaunchKernelGGL(k_merge_norms<F32In>, dim3(parts, (unsigned)d.BH), dim3(kMergeThreads), 0, st,
                         (const float*)Q, (const float*)K, belong, centroid, d.n, d.N, rad2g, qmax2g);
  }
  TimedLaunch tl("merge_pairs", st);
  hipLaunchKernelGGL(k_merge_pairs, dim3((unsigned)d.BH), dim3(kMergeThreads), 0, st, centroid, count, d.N,
                     abs_scale, log_eps, radius, dthr, partner, merges);
  return hipGetLastError();
}

}  // namespace ga
