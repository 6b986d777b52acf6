// gfx950 (MI355X) kernels for RITA group attention.
//
// Grouping (Section 4.4): Lloyd K-means on the keys of every (b, h) slice, the
// squared distance expanded as |r|^2 - 2 k.r so that its bulk is the n x N x d
// contraction K R^T.  Aggregation and group softmax: Section 4.2, Eq. 3,
// Algorithm 1.
//
// Kernels, in the order the forward runs them (bf16, N <= 128):
//   k_assign_reg<true, NB, true>   first round: initial centroids C0_j =
//                   k_{floor(j n / N)} (or a given init), R = round(C), the
//                   canonical fp64 |r_j|^2; MFMA 32x32x16 bf16 scores
//                   |r_j|^2 - 2 k.r_j with an in-register top-2 per key; keys
//                   whose top-2 gap is inside a rigorous error band are
//                   re-decided with the exact fp64 definition; then the
//                   workgroup's fp64 partition of the group sums
//   k_part_finish   adds the partitions: counts, C, R, |r|^2
//   k_assign_reg<false, NB, false> + k_gdelta   each later round: the same
//                   assignment, then the member sums of the groups changed by
//                   the moved keys only
//   k_gsum<3>       value sums, written as the attention's bf16 value means
//                   (transposed) and log2(count) score bias
//   k_attend_bf16   MFMA scores, block-wise group softmax, MFMA combine
// Also: k_init, k_assign_bf16 (N <= 1024), k_gsum<0> (first-round sums
// without partitions), k_gsum<2> (value sums), k_attend_prep; the fp32 path
// k_assign_exact (fp64 fma-chain scores for every (key, group)), k_bucket
// (stable counting sort of keys by group), k_segsum (one wave per group sums
// its members in ascending key order in fp64) and k_attend_f32.
#include <hip/hip_runtime.h>

#include <float.h>
#include <math.h>
#include <stdint.h>

#include <map>
#include <mutex>
#include <tuple>

#include "ga_internal.h"

namespace ga {
namespace {

#include "ga_device.h"


constexpr int kRs = 72;       // LDS row stride (bf16 elements) of the 32x16 MFMA A tiles
constexpr int kAttDepth = 2;     // query tiles loaded ahead per wave in k_attend_bf16
constexpr int kOs = 72;          // LDS row stride (bf16) of the attention output tiles
constexpr int kExactB = 4;       // queued keys decided together by one wave in k_assign_reg
constexpr int kAttMaxN = 256; // groups held in LDS by the bf16 attention kernel

// Representative of one group row from its fp32 centroid value (lane = feature).
template <class S>
__device__ void finalize_rep(float c, int64_t row, typename S::T* R, double* nrm64, uint16_t* nsplit) {
  const int lane = threadIdx.x & 63;
  const float r = S::rep(c);
  S::store(R, row * 64 + lane, r);
  const double nrm = canon_nrm_wave(r);
  if (lane == 0) {
    nrm64[row] = nrm;
    write_nsplit(nrm, nsplit + row * 8);
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
// grid (ceil(N/64), BH), 256 threads; groups g0 = 64 x .. g0 + 63.  Each wave
// reads 16 groups' initial rows at once (lane = feature) and writes C and R;
// then one lane per group forms the canonical |r|^2 from the LDS copy of R.
template <class S>
__global__ __launch_bounds__(256) void k_init(const typename S::T* __restrict__ K,
                                              const float* __restrict__ init, int n, int N,
                                              float* __restrict__ C, typename S::T* __restrict__ R,
                                              double* __restrict__ nrm64, uint16_t* __restrict__ nsplit,
                                              int32_t* __restrict__ mcount) {
  __shared__ float rsh[64][65];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t bh = blockIdx.y;
  const int g0 = blockIdx.x * 64, ng = min(64, N - g0);
  float c[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int g = min(g0 + wave * 16 + i, N - 1);
    const int64_t row = bh * N + g;
    c[i] = init ? init[row * 64 + lane] : S::load(K, (bh * n + ((int64_t)g * n) / N) * 64 + lane);
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int gl = wave * 16 + i;
    if (gl >= ng) break;
    const int64_t row = bh * N + g0 + gl;
    C[row * 64 + lane] = c[i];
    const float r = S::rep(c[i]);
    S::store(R, row * 64 + lane, r);
    rsh[gl][lane] = r;
  }
  if (mcount && blockIdx.x == 0 && tid == 0) {
    mcount[bh] = 0;
    mcount[gridDim.y + bh] = 0;
  }
  __syncthreads();
  if (tid < ng) {
    const int64_t row = bh * N + g0 + tid;
    double nrm = 0.0;
#pragma unroll 8
    for (int cc = 0; cc < 64; ++cc) {
      const double rc = (double)rsh[tid][cc];
      nrm = fma(rc, rc, nrm);
    }
    nrm64[row] = nrm;
    write_nsplit(nrm, nsplit + row * 8);
  }
}

// ------------------------------------------------------------------ assign (bf16, MFMA)




// Per-workgroup state of the assign kernels, in LDS.  Keys are numbered
// locally within the workgroup (lk < 4 tpw 32 <= 2048, 11 bits; groups < 1024,
// 10 bits).  The groups (and in the first round the |k| bounds) are staged
// here and written out once at the end, so the scoring loop issues no global
// stores and the only memory operations between a tile's prefetch and its use
// are the unconditional loads of the next tile (which keeps the compiler's
// wait counts exact).  Each wave appends moved keys and uncertain keys to its
// own region of tpw 32 entries with a wave-uniform counter (no atomics).
struct AssignCounts {
  int wcnt[4], ucnt[4];  // per-wave moved / uncertain entries
  int nx, moved_base;    // moved keys found by the exact decisions
};
struct AssignLists {
  AssignCounts* c;
  uint32_t* wrec;  // [4][tpw 32] moved keys: lk | old << 11 | new << 21
  uint32_t* uq;    // [4][tpw 32] uncertain keys: lk | old << 11
  int32_t* bst;    // [4 tpw 32] group of every local key
  uint32_t* kx;    // [4 tpw 32] first round: |k| bounds (float bits); later: moved keys of the exact decisions
  int cap;         // tpw 32
};


// Decision for the keys of two tiles A and B at once, given each lane's top-2
// over its half of the groups for both: one lane swap per value leaves lane
// q < 32 with both halves of key q of A and lane 32 + q with both halves of
// key q of B, so every lane decides one key.  The lane merges its halves,
// certifies the packed best against the error bound E, stages the group and
// (later rounds) records keys whose group changed.  Keys that fail the test
// are queued for exact_decide_queue (their staged group is provisional).
// knv, oldv, lk: the lane's own key; stage: its tile exists (for B possibly
// not, after an odd tile count); valid: also a key below n.
//
// E bounds |packed - exact| for the best and for any group that could beat
// it: the MFMA part cm * M (M = max |r|^2 + 2 |k| max |r| bounds the sum of
// |terms|) and the packing part cp * (|M1| + 3 cm M); the last two terms cover
// the fp32 evaluation of E and of M1 + 2E.
template <bool FIRST>
__device__ __forceinline__ void decide_pair(float M1a, float M2a, int B1a, float M1b, float M2b, int B1b, float knv,
                                            int oldv, int lk, bool stage, bool valid, int N, const Certify& cf,
                                            const AssignLists& sh, int wave, int& wn, int& un) {
  const auto p1 = __builtin_amdgcn_permlane32_swap(__float_as_uint(M1a), __float_as_uint(M1b), false, false);
  const auto p2 = __builtin_amdgcn_permlane32_swap(__float_as_uint(M2a), __float_as_uint(M2b), false, false);
  const auto pb = __builtin_amdgcn_permlane32_swap((uint32_t)B1a, (uint32_t)B1b, false, false);
  // [0]: the best over the groups held by lanes 0-31, [1]: by lanes 32-63
  const float a1 = __uint_as_float(p1[0]), b1 = __uint_as_float(p1[1]);
  // the half held by lanes 32-63 wins only with a strictly smaller best
  const bool hi_wins = b1 < a1;
  const uint32_t vw = __float_as_uint(hi_wins ? b1 : a1) & kPackMask;
  const int jstar = 32 * (int)(hi_wins ? pb[1] : pb[0]) + 8 * (int)(vw >> 2) + (hi_wins ? 4 : 0) + (int)(vw & 3);
  const float best = min2(a1, b1);
  const float second = min2(max2(a1, b1), min2(__uint_as_float(p2[0]), __uint_as_float(p2[1])));
  const float Mk = cf.nmaxf + 2.0f * knv * cf.rmaxf;
  const float aM1 = fabsf(best);
  const float E = (cf.cm * Mk + cf.cp * (aM1 + 3.0f * cf.cm * Mk)) * (1.0f + 0x1p-20f) + 0x1p-22f * aM1 + 1e-30f;
  const bool certain = (second > best + 2.0f * E) && (jstar < N);
  if (stage) sh.bst[lk] = jstar;
  wave_append(valid && !certain, (uint32_t)lk | ((uint32_t)oldv << 11), sh.uq + wave * sh.cap, un);
  if (!FIRST)
    wave_append(valid && certain && oldv != jstar,
                (uint32_t)lk | ((uint32_t)oldv << 11) | ((uint32_t)jstar << 21), sh.wrec + wave * sh.cap, wn);
}

// Entry u of the concatenation of four per-wave regions with counts cnt[0..3].
__device__ __forceinline__ uint32_t region_entry(const uint32_t* base, int cap, const int* cnt, int u) {
  int r = 0;
  while (r < 3 && u >= cnt[r]) u -= cnt[r++];
  return base[r * cap + u];
}

// After every tile of the workgroup is scored: each wave takes a quarter of
// the queued keys (consecutive entries) and decides them B at a time
// with exact_argmin_keys (their rows widened to fp64 in the wave's LDS slot
// kd_w, [B][64]), then stages and records each like decide_pair.
template <bool FIRST, int B>
__device__ __forceinline__ void exact_decide_queue(const uint16_t* __restrict__ Kbh, int64_t key0, const uint16_t* Rs,
                                                   const double* __restrict__ nrm_bh, int N, double* kd_w,
                                                   const AssignLists& sh, int nunc) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int per = (nunc + 3) >> 2;
  const int u_end = min(nunc, (wave + 1) * per);
  for (int u0 = wave * per; u0 < u_end; u0 += B) {
    const int nb = min(B, u_end - u0);
    uint32_t e[B];
#pragma unroll
    for (int b = 0; b < B; ++b) {
      e[b] = b < nb ? region_entry(sh.uq, sh.cap, sh.c->ucnt, u0 + b) : 0u;
      if (b < nb) kd_w[b * 64 + lane] = (double)bf16_to_f32(Kbh[(key0 + (e[b] & 2047u)) * 64 + lane]);
    }
    int jb[B];
    switch (nb) {  // wave-uniform
      case 1: exact_argmin_keys<1>(kd_w, Rs, nrm_bh, N, jb); break;
      case 2: exact_argmin_keys<(B >= 2 ? 2 : 1)>(kd_w, Rs, nrm_bh, N, jb); break;
      case 3: exact_argmin_keys<(B >= 3 ? 3 : 1)>(kd_w, Rs, nrm_bh, N, jb); break;
      default: exact_argmin_keys<B>(kd_w, Rs, nrm_bh, N, jb); break;
    }
    if (lane == 0) {
#pragma unroll
      for (int b = 0; b < B; ++b) {
        if (b >= nb) break;
        const int lk = (int)(e[b] & 2047u), oldv = (int)(e[b] >> 11);
        sh.bst[lk] = jb[b];
        if (!FIRST && oldv != jb[b])
          sh.kx[atomicAdd(&sh.c->nx, 1)] = (uint32_t)lk | ((uint32_t)oldv << 11) | ((uint32_t)jb[b] << 21);
      }
    }
  }
}

// Stage -2R (swizzled, see swz) and the |r|^2 split of one slice into LDS and
// return the slice's largest canonical |r|^2.  Padded groups (j >= N) get
// zero rows and the largest bf16 as |r|^2, so they never win.  Every thread
// issues all of its loads before converting (NPAD_C > 0: Npad known at
// compile time).  Ends with a barrier.
template <int NPAD_C>
__device__ __forceinline__ double stage_reps(const uint16_t* __restrict__ Rbh, const uint16_t* __restrict__ nsplit_bh,
                                             const double* __restrict__ nrm_bh, int N, int Npad_rt, uint16_t* Rs,
                                             uint16_t* Ns, double* red) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int Npad = NPAD_C > 0 ? NPAD_C : Npad_rt;
  const int j = tid;  // Npad <= 1024 rows: the split and |r|^2 of rows tid, tid + 256, ...
  u32x4 sp = {0x7f7fu, 0u, 0u, 0u};
  double mx = 0.0;
  if (j < N) {
    sp = *(const u32x4*)(nsplit_bh + j * 8);
    mx = nrm_bh[j];
  }
  if (NPAD_C > 0) {
    constexpr int IT = NPAD_C > 0 ? NPAD_C * 8 / 256 : 1;
    u32x4 w[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = tid + it * 256, row = idx >> 3, ch = idx & 7;
      w[it] = row < N ? *(const u32x4*)(Rbh + (int64_t)row * 64 + ch * 8) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = tid + it * 256, row = idx >> 3, ch = idx & 7;
      u32x4 v;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t lo = __float_as_uint(bf16_to_f32(w[it][e] & 0xffffu) * -2.0f) >> 16;
        const uint32_t hi = __float_as_uint(bf16_to_f32(w[it][e] >> 16) * -2.0f) >> 16;
        v[e] = lo | (hi << 16);
      }
      *(u32x4*)(Rs + swz(row, ch)) = v;
    }
  } else {
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
      *(u32x4*)(Rs + swz(row, ch)) = v;
    }
  }
  if (j < Npad) *(u32x4*)(Ns + j * 8) = sp;
  for (int jj = tid + 256; jj < Npad; jj += 256) {
    const u32x4 sp2 = jj < N ? *(const u32x4*)(nsplit_bh + jj * 8) : u32x4{0x7f7fu, 0u, 0u, 0u};
    *(u32x4*)(Ns + jj * 8) = sp2;
    if (jj < N) mx = fmax(mx, nrm_bh[jj]);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mx = fmax(mx, __shfl_xor(mx, off));
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  return fmax(fmax(red[0], red[1]), fmax(red[2], red[3]));
}

// First round with partition sums: the initial representatives straight from
// the keys (C_j = k_{floor(j n / N)}, R = C) or from a given init (C_j =
// init_j, R = bf16(C)), staged like stage_reps, without a separate init
// launch.  The canonical |r|^2 (fma chain over c = 0..63, one thread per
// group) goes to nrm_l and its split to Ns; C_bh, if given, receives C.  Ends
// with a barrier; returns the slice's largest |r|^2.
template <int NPAD>
__device__ __forceinline__ double stage_init(const uint16_t* __restrict__ Kbh, const float* __restrict__ init_bh,
                                             int n, int N, float* __restrict__ C_bh, uint16_t* Rs, uint16_t* Ns,
                                             double* nrm_l, double* red) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int IT = NPAD * 8 / 256;
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int idx = tid + it * 256, row = idx >> 3, ch = idx & 7;
    u32x4 r = {0u, 0u, 0u, 0u};
    if (row < N) {
      float c[8];
      if (init_bh) {
        const float4 a = *(const float4*)(init_bh + row * 64 + ch * 8);
        const float4 b = *(const float4*)(init_bh + row * 64 + ch * 8 + 4);
        c[0] = a.x; c[1] = a.y; c[2] = a.z; c[3] = a.w; c[4] = b.x; c[5] = b.y; c[6] = b.z; c[7] = b.w;
#pragma unroll
        for (int e = 0; e < 4; ++e) r[e] = f32_to_bf16(c[2 * e]) | (f32_to_bf16(c[2 * e + 1]) << 16);
      } else {
        r = *(const u32x4*)(Kbh + ((int64_t)row * n / N) * 64 + ch * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          c[2 * e] = bf16_to_f32(r[e] & 0xffffu);
          c[2 * e + 1] = bf16_to_f32(r[e] >> 16);
        }
      }
      if (C_bh) {
        *(float4*)(C_bh + row * 64 + ch * 8) = float4{c[0], c[1], c[2], c[3]};
        *(float4*)(C_bh + row * 64 + ch * 8 + 4) = float4{c[4], c[5], c[6], c[7]};
      }
    }
    u32x4 v;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t lo = __float_as_uint(bf16_to_f32(r[e] & 0xffffu) * -2.0f) >> 16;
      const uint32_t hi = __float_as_uint(bf16_to_f32(r[e] >> 16) * -2.0f) >> 16;
      v[e] = lo | (hi << 16);
    }
    *(u32x4*)(Rs + swz(row, ch)) = v;
  }
  __syncthreads();
  double mx = 0.0;
  if (tid < NPAD) {
    const int j = tid;
    double nrm = 0.0;
    if (j < N) {
#pragma unroll
      for (int ch = 0; ch < 8; ++ch) {
        const u32x4 v = *(const u32x4*)(Rs + swz(j, ch));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const double lo = (double)(-0.5f * bf16_to_f32(v[e] & 0xffffu));
          const double hi = (double)(-0.5f * bf16_to_f32(v[e] >> 16));
          nrm = fma(lo, lo, nrm);
          nrm = fma(hi, hi, nrm);
        }
      }
      write_nsplit(nrm, Ns + j * 8);
      mx = nrm;
    } else {
      *(u32x4*)(Ns + j * 8) = u32x4{0x7f7fu, 0u, 0u, 0u};
    }
    nrm_l[j] = nrm;
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mx = fmax(mx, __shfl_xor(mx, off));
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  return fmax(fmax(red[0], red[1]), fmax(red[2], red[3]));
}

// Dynamic LDS of the assign kernels: region A = -2R as [Npad][64] bf16
// (swizzled), the |r|^2 split as [Npad][8] bf16 and the uncertain queue
// (4 tpw 32 words), then three arrays of 4 tpw 32 words: moved records, staged
// groups, staged |k| bounds / exact-decision moved records.  Region A is dead
// once the exact decisions are done; the partition sums reuse it (and need it
// at least fused_bytes(...) long).
// Partition sums: the sorted key list (groups padded to 8) then four
// per-wave [8][64] fp64 transpose tiles.
__host__ __device__ constexpr int fused_words(int Npad, int cap4) { return (cap4 + 7 * Npad + 3) & ~3; }
__host__ __device__ constexpr int fused_bytes(int Npad, int cap4) { return fused_words(Npad, cap4) * 4 + 4 * 4096; }
__host__ __device__ constexpr int assign_region_a(int Npad, int cap4, bool fused) {
  return fused && fused_bytes(Npad, cap4) > Npad * 144 + cap4 * 4 ? fused_bytes(Npad, cap4) : Npad * 144 + cap4 * 4;
}

struct AssignLds {
  uint16_t* Rs;
  uint16_t* Ns;
  AssignLists lists;
};

__device__ __forceinline__ AssignLds assign_lds_layout(unsigned char* smem, int Npad, int tpw, bool fused,
                                                       AssignCounts* c) {
  const int cap = tpw * 32;
  AssignLds l;
  l.Rs = (uint16_t*)smem;
  l.Ns = l.Rs + Npad * 64;
  l.lists.c = c;
  l.lists.cap = cap;
  l.lists.uq = (uint32_t*)(l.Ns + Npad * 8);
  l.lists.wrec = (uint32_t*)(smem + assign_region_a(Npad, 4 * cap, fused));
  l.lists.bst = (int32_t*)(l.lists.wrec + 4 * cap);
  l.lists.kx = (uint32_t*)(l.lists.bst + 4 * cap);
  return l;
}

// End of an assign workgroup (after each wave stored its counts): exact
// decisions of the queued keys, then the staged groups (and first-round |k|
// bounds) of keys key0 .. key0 + 4 tpw 32 (those below n); without the fused
// update also the moved-key records, one global atomic per workgroup.
template <bool FIRST, bool FUSED, int B>
__device__ __forceinline__ void assign_epilogue(const uint16_t* __restrict__ Kbh, int64_t key0, int tpw,
                                                const uint16_t* Rs, const double* nrm_bh, int n, int N,
                                                int32_t* __restrict__ belong_bh, float* __restrict__ knorm_bh,
                                                int32_t* __restrict__ mcount_bh,
                                                unsigned long long* __restrict__ mrec_bh, double* kd_w,
                                                const AssignLists& sh) {
  const int tid = threadIdx.x;
  __syncthreads();
  const int* uc = sh.c->ucnt;
  const int nunc = uc[0] + uc[1] + uc[2] + uc[3];
  if (nunc) {  // uniform: read after the barrier
    exact_decide_queue<FIRST, B>(Kbh, key0, Rs, nrm_bh, N, kd_w, sh, nunc);
    __syncthreads();
  }
  // the first round writes every key's group; later rounds only those of the
  // keys that moved (the others keep theirs)
  if (FIRST) {
    const int nk = (int)min((int64_t)4 * tpw * 32, (int64_t)n - key0);
    for (int x = tid; x < nk; x += 256) {
      belong_bh[key0 + x] = sh.bst[x];
      knorm_bh[key0 + x] = __uint_as_float(sh.kx[x]);
    }
  }
  if (!FIRST && !FUSED) {
    const int* wc = sh.c->wcnt;
    const int nw = wc[0] + wc[1] + wc[2] + wc[3];
    const int nm = nw + sh.c->nx;
    if (tid == 0) sh.c->moved_base = nm ? atomicAdd(mcount_bh, nm) : 0;
    __syncthreads();
    // a slice records at most n moved keys in a round; the bound only guards
    // against a counter that was not cleared (a corrupted workspace)
    const int base = sh.c->moved_base;
    for (int x = tid; x < nm; x += 256) {
      const uint32_t e = x < nw ? region_entry(sh.wrec, sh.cap, wc, x) : sh.kx[x - nw];
      belong_bh[key0 + (e & 2047u)] = (int32_t)(e >> 21);
      if ((int64_t)base + x < n)
        mrec_bh[base + x] = ((unsigned long long)(key0 + (e & 2047u)) << 32) | (((e >> 11) & 1023u) << 16) |
                            (e >> 21);
    }
  }
}

// ------------------------------------------------------------------ exact sums (bf16)
// With bf16 keys and values every fp64 member sum is exact: a member is a
// multiple of 2^(e_min - 7) (8-bit significand, e_min the smallest member
// exponent) and every partial sum, in any order, is below 2^(e_max + 1 +
// log2 count), so all of them are representable in fp64's 53 bits whenever
// (e_max - e_min) + log2 count <= 45, e.g. at most 2^15 members with nonzero
// magnitudes within 2^30 of each other.  The order of summation then cannot
// change a bit, and the bf16 path sums without a stable order.

constexpr int kGsumU = 8;        // 8-row chunks per batch

// One batch of a wave's run: entries of chunks ch0 .. ch0 + U - 1 (clamped
// to the run's last chunk, so every lane loads) and their row fragments.
template <int U>
__device__ __forceinline__ void gsum_load(const uint32_t* ent, const uint16_t* __restrict__ Xb, int ch0, int ce,
                                          int slot, int j, uint32_t (&e)[U], u32x4 (&w)[U]) {
#pragma unroll
  for (int u = 0; u < U; ++u) {
    e[u] = ent[min(ch0 + u, ce - 1) * 8 + slot];
    const uint32_t key = e[u] == 0xffffffffu ? 0u : (e[u] & 0x7fffffffu);
    w[u] = *(const u32x4*)(Xb + (int64_t)key * 64 + 8 * j);
  }
}

// ------------------------------------------------------------------ partition sums (bf16, N <= 128)
// The member sums of the bf16 path are exact in fp64 (see above), so they may
// be split into per-workgroup partitions and added in any order.  In the first
// round, after its decisions, assign workgroup p of slice bh (keys key0 ..
// key0 + nk - 1) sorts its keys by group in LDS; each wave sums the rows of a
// run of whole groups in fp64 registers (8 rows per instruction, 16 bytes per
// lane) and stores each finished group's row into partition p of Sp, together
// with the member counts and a bitmask of the groups with members.
// k_part_finish then adds the partitions.  (Later rounds move few keys; there
// a separate launch over the moved-key records is faster than lengthening
// every assign workgroup by its share of the sums.)
struct PartLds {
  int ecnt[kFusedG], eoff[kFusedG + 1], ecur[kFusedG], wbeg[5], wg0[4];
};

__device__ __forceinline__ void partition_sums(const uint16_t* __restrict__ Kbh, int64_t key0, int nk, int N,
                                               const AssignLists& sh, uint32_t* ent, int tw_words, PartLds& fl,
                                               const FusedUpdate& fu) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t bh = blockIdx.y;
  const int p = (int)blockIdx.x;
  if (tid < kFusedG) fl.ecnt[tid] = 0;
  __syncthreads();
  for (int x = tid; x < nk; x += 256) atomicAdd(&fl.ecnt[sh.bst[x]], 1);
  __syncthreads();
  // layout (wave 0, groups 2 lane and 2 lane + 1): each group's keys padded
  // to a multiple of 8; wave w takes the groups from the first one starting at
  // or after w tot / 4
  if (wave == 0) {
    const int ga = 2 * lane, gb = ga + 1;
    const int ca = fl.ecnt[ga], cb = fl.ecnt[gb];
    const int pa = (ca + 7) & ~7, pb = (cb + 7) & ~7;
    int incl = pa + pb;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int y = __shfl_up(incl, off);
      if (lane >= off) incl += y;
    }
    const int sa = incl - pa - pb, sb = sa + pa, tot = __shfl(incl, 63);
    fl.eoff[ga] = sa;
    fl.eoff[gb] = sb;
    fl.ecur[ga] = sa;
    fl.ecur[gb] = sb;
    for (int k = ca; k < pa; ++k) ent[sa + k] = 0xffffffffu;
    for (int k = cb; k < pb; ++k) ent[sb + k] = 0xffffffffu;
    if (lane == 0) {
      fl.eoff[kFusedG] = tot;
      fl.wbeg[0] = 0;
      fl.wbeg[4] = tot;
      fl.wg0[0] = 0;
    }
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      const int thr = w * tot / 4;
      // the starts grow with g: the groups starting before thr are a prefix
      const int g = (int)__popcll(__ballot(sa < thr)) + (int)__popcll(__ballot(sb < thr));
      const int gsa = __shfl(sa, (g >> 1) & 63), gsb = __shfl(sb, (g >> 1) & 63);
      if (lane == 0) {
        fl.wbeg[w] = g < kFusedG ? ((g & 1) ? gsb : gsa) : tot;
        fl.wg0[w] = g;
      }
    }
    const uint64_t t0 = __ballot(fl.ecnt[lane] > 0), t1 = __ballot(fl.ecnt[lane + 64] > 0);
    if (lane < 4) fu.pbits[(bh * kFusedP + p) * 4 + lane] = (uint32_t)((lane < 2 ? t0 : t1) >> (32 * (lane & 1)));
  }
  __syncthreads();
  for (int x = tid; x < nk; x += 256) ent[atomicAdd(&fl.ecur[sh.bst[x]], 1)] = (uint32_t)x;
  if (tid < N) fu.cntp[(bh * kFusedP + p) * N + tid] = fl.ecnt[tid];
  __syncthreads();
  // per-wave register sums over runs of whole groups into partition p
  const int slot = lane >> 3, j = lane & 7;
  const int cb = fl.wbeg[wave] / 8, ce = fl.wbeg[wave + 1] / 8;
  const uint16_t* Xb = Kbh + key0 * 64;
  double* Spp = fu.Sp + (bh * kFusedP + p) * (int64_t)N * 64;
  // per-wave [8 slots][64 features] transpose tile after the entry list: the
  // 8 slot rows of a finished group are added by lane = feature and stored as
  // one row
  double* tw = (double*)(ent + tw_words) + wave * 512;
  double a[8] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
  int g = fl.wg0[wave], gend = 0;  // current group and its end chunk
  auto flush = [&]() {
#pragma unroll
    for (int k = 0; k < 8; k += 2) *(double2*)(tw + slot * 64 + 8 * j + k) = double2{a[k], a[k + 1]};
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    double v = tw[lane];
#pragma unroll
    for (int k = 1; k < 8; ++k) v += tw[k * 64 + lane];
    Spp[g * 64 + lane] = v;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int k = 0; k < 8; ++k) a[k] = 0.0;
  };
  auto add = [&](int ch0, const uint32_t (&e)[kGsumU], const u32x4 (&w)[kGsumU]) {
#pragma unroll
    for (int u = 0; u < kGsumU; ++u) {
      const int ch = ch0 + u;
      if (ch >= ce) break;
      if (ch >= gend) {  // next non-empty group (uniform)
        if (ch > cb) flush();
        while (fl.eoff[g + 1] <= ch * 8) ++g;
        gend = fl.eoff[g + 1] / 8;
      }
      const double sg = e[u] == 0xffffffffu ? 0.0 : 1.0;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const uint32_t bits = (k & 1) ? (w[u][k >> 1] >> 16) : (w[u][k >> 1] & 0xffffu);
        a[k] = fma(sg, (double)bf16_to_f32(bits), a[k]);
      }
    }
  };
  if (cb < ce) {
    uint32_t eA[kGsumU], eB[kGsumU];
    u32x4 wA[kGsumU], wB[kGsumU];
    gsum_load(ent, Xb, cb, ce, slot, j, eA, wA);
    for (int ch0 = cb; ch0 < ce; ch0 += 2 * kGsumU) {
      gsum_load(ent, Xb, ch0 + kGsumU, ce, slot, j, eB, wB);
      __builtin_amdgcn_sched_barrier(0);
      add(ch0, eA, wA);
      if (ch0 + kGsumU >= ce) break;
      gsum_load(ent, Xb, ch0 + 2 * kGsumU, ce, slot, j, eA, wA);
      __builtin_amdgcn_sched_barrier(0);
      add(ch0 + kGsumU, eB, wB);
    }
    flush();
  }
}

// k_part_finish: grid (ceil(N / 32), BH), 256 threads; after a first-round
// assign launch with partition sums (P partitions per slice).  Workgroup x
// finishes groups g0 = 32 x .. g0 + 31 of slice bh: S64 = the sum over the
// partitions with members of the group, count = their member counts, C =
// (float)(S / count) (an empty group keeps C), R = bf16(C), the canonical fp64
// |r|^2 (fma chain over c = 0..63, one lane per group) and its split.  Thread
// t adds features 2 (t % 32), +1 of groups g0 + t / 32 + 8 u; only the rows of
// (partition, group) pairs with members are read, all at once.
template <int P>
__global__ __launch_bounds__(256) void k_part_finish(const double* __restrict__ Sp, const int32_t* __restrict__ cntp,
                                                     const uint32_t* __restrict__ pbits, int N,
                                                     double* __restrict__ S64, int32_t* __restrict__ count,
                                                     float* __restrict__ C, uint16_t* __restrict__ R,
                                                     double* __restrict__ nrm64, uint16_t* __restrict__ nsplit) {
  __shared__ uint32_t tb[P];  // bit g - g0: partition q has members of group g
  __shared__ int ctl[P][32];
  __shared__ uint32_t rsh[32][33];  // R rows as bf16 pairs
  const int tid = threadIdx.x;
  const int64_t bh = blockIdx.y;
  const int g0 = blockIdx.x * 32, ng = min(32, N - g0);
  if (tid < P * 32) {
    const int q = tid >> 5, g = tid & 31;
    const int cv = cntp[(bh * kFusedP + q) * N + g0 + min(g, ng - 1)];
    const uint32_t bw = pbits[(bh * kFusedP + q) * 4 + (g0 >> 5)];
    ctl[q][g] = cv;
    if (g == 0) tb[q] = bw;
  }
  const int c2 = tid & 31, gq = tid >> 5;
  const int64_t row0 = bh * N;
  double2 sacc[4];
  int pcnt[4];
  f32x2 cold[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int gc = g0 + min(gq + 8 * u, ng - 1);
    sacc[u] = double2{0.0, 0.0};
    pcnt[u] = 0;
    cold[u] = *(const f32x2*)(C + (row0 + gc) * 64 + 2 * c2);
  }
  __syncthreads();
  double2 v[4][P];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int g = gq + 8 * u, gc = g0 + min(g, ng - 1);
#pragma unroll
    for (int q = 0; q < P; ++q) {
      const bool hit = (tb[q] >> g) & 1u;
      v[u][q] = hit ? *(const double2*)(Sp + ((bh * kFusedP + q) * N + gc) * 64 + 2 * c2) : double2{0.0, 0.0};
    }
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int g = gq + 8 * u;
#pragma unroll
    for (int q = 0; q < P; ++q) {
      sacc[u].x += v[u][q].x;
      sacc[u].y += v[u][q].y;
      pcnt[u] += ((tb[q] >> g) & 1u) ? ctl[q][g] : 0;
    }
    if (g >= ng) continue;
    const int64_t row = row0 + g0 + g;
    *(double2*)(S64 + row * 64 + 2 * c2) = sacc[u];
    if (c2 == 0) count[row] = pcnt[u];
    f32x2 cf = cold[u];
    if (pcnt[u] > 0) {
      cf.x = (float)(sacc[u].x / (double)pcnt[u]);
      cf.y = (float)(sacc[u].y / (double)pcnt[u]);
      *(f32x2*)(C + row * 64 + 2 * c2) = cf;
    }
    const uint32_t rp = f32_to_bf16(cf.x) | (f32_to_bf16(cf.y) << 16);
    *(uint32_t*)(R + row * 64 + 2 * c2) = rp;
    rsh[g][c2] = rp;
  }
  __syncthreads();
  if (tid < ng) {
    double nrm = 0.0;
#pragma unroll 8
    for (int c = 0; c < 64; ++c) {
      const uint32_t w = rsh[tid][c >> 1];
      const double rc = (double)bf16_to_f32((c & 1) ? (w >> 16) : (w & 0xffffu));
      nrm = fma(rc, rc, nrm);
    }
    nrm64[row0 + g0 + tid] = nrm;
    write_nsplit(nrm, nsplit + (row0 + g0 + tid) * 8);
  }
}

// MFMA 32x32x16 scoring shared by both assign kernels: rows = 32 groups
// (A = -2R), columns = 32 keys (B = K).  Lane l (h = l/32, q = l%32) supplies
// at k-step s features 32h + 8s .. +7 of its row for both operands (the same
// permutation of the contraction axis on both sides) and receives groups
// 8(v/4) + 4h + v%4 of key q in accumulator register v.  A fifth k-step adds
// |r_j|^2 = hi + mid + lo (A = the split, B = ones in the first three slots
// of lanes h = 0), so each output is the score s_ij = |r_j|^2 - 2 k_i.r_j.
//
// If second - best > 2E, where E bounds |packed - exact| (the MFMA fp32
// accumulation, the split of |r|^2 and the packing), the packed best is
// provably the exact fp64 argmin; otherwise the key is queued and re-decided
// by exact_argmin_keys once the workgroup's tiles are done.  Later rounds
// (FIRST = false) also emit the keys whose group changed as records
// (key, old, new).
//
// k_assign_bf16: grid (ceil(tiles / (4 * tpw)), BH), 256 threads, any N up to
// 1024 (k_assign_reg covers N <= 128).  Each wave owns tpw consecutive 32-key
// tiles and scores them two at a time (two independent MFMA / VALU chains
// sharing the A-operand reads, which come from LDS); the next pair's key
// fragments are loaded while the current pair is scored.
template <bool FIRST>
__global__ __launch_bounds__(256) void k_assign_bf16(
    const uint16_t* __restrict__ K, const uint16_t* __restrict__ R, const uint16_t* __restrict__ nsplit,
    const double* __restrict__ nrm64, float* __restrict__ knorm, int32_t* __restrict__ belong,
    int32_t* __restrict__ mcount, unsigned long long* __restrict__ mrec, int n, int N, int tpw, float cm,
    float cp, FusedUpdate) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ double red[4];
  __shared__ AssignCounts cnt;
  __shared__ __align__(16) double kd[4][64];  // fp64 row of a queued key, per wave
  const int Npad = (N + 31) & ~31;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5, q = lane & 31;
  const int64_t bh = blockIdx.y;
  if (tid == 0) cnt.nx = 0;
  const AssignLds L = assign_lds_layout(smem, Npad, tpw, false, &cnt);
  const uint16_t* Rs = L.Rs;
  const uint16_t* Ns = L.Ns;
  const double nmax = stage_reps<0>(R + bh * (int64_t)N * 64, nsplit + bh * N * 8, nrm64 + bh * N, N, Npad, L.Rs,
                                    L.Ns, red);
  const float nmaxf = (float)nmax * (1.0f + 0x1p-20f);
  const float rmaxf = sqrtf(nmaxf) * (1.0f + 0x1p-20f);
  const Certify cf = {nmaxf, rmaxf, cm, cp};

  const int nblk = Npad >> 5;
  const int64_t key0 = (int64_t)blockIdx.x * 4 * tpw * 32;
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const int64_t tile0 = key0 / 32 + (int64_t)wv * tpw;
  const int64_t ntiles = ((int64_t)n + 31) / 32;
  const int tcount = (int)max((int64_t)0, min((int64_t)tpw, ntiles - tile0));
  const uint16_t* Kbh = K + bh * (int64_t)n * 64;
  const float* knorm_bh = knorm + bh * n;
  int32_t* belong_bh = belong + bh * n;
  // B operand of the |r|^2 k-step: ones in the first three slots of lanes h = 0
  const u32x4 ones = h == 0 ? u32x4{0x3f803f80u, 0x3f80u, 0u, 0u} : u32x4{0u, 0u, 0u, 0u};
  const f32x16 zero = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};

  int wn = 0, un = 0;  // this wave's moved / uncertain entries (wave-uniform)
  u32x4 kf[2][4];
  float kn[2] = {0.f, 0.f};
  int old[2] = {0, 0};
  auto fetch = [&](int t, u32x4 (&f)[4], float& knv, int& oldv) {
    const int64_t key = (tile0 + t) * 32 + q;
    const bool valid = t < tcount && key < n;
    const uint16_t* krow = Kbh + (valid ? key : 0) * 64 + h * 32;
#pragma unroll
    for (int s2 = 0; s2 < 4; ++s2) f[s2] = valid ? *(const u32x4*)(krow + s2 * 8) : u32x4{0u, 0u, 0u, 0u};
    if (!FIRST) {
      knv = valid ? knorm_bh[key] : 0.f;
      oldv = valid ? belong_bh[key] : 0;
    }
  };
  if (tcount > 0) {
    fetch(0, kf[0], kn[0], old[0]);
    fetch(1, kf[1], kn[1], old[1]);
  }

  for (int tt = 0; tt < tcount; tt += 2) {
    u32x4 kf_n[2][4];
    float kn_n[2] = {0.f, 0.f};
    int old_n[2] = {0, 0};
    if (tt + 2 < tcount) {
      fetch(tt + 2, kf_n[0], kn_n[0], old_n[0]);
      fetch(tt + 3, kf_n[1], kn_n[1], old_n[1]);
    }
    bool valid[2];
    int lk[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      lk[u] = (wv * tpw + tt + u) * 32 + q;
      valid[u] = tt + u < tcount && key0 + lk[u] < n;
      if (FIRST) {
        kn[u] = key_norm_bound(kf[u]);
        if (tt + u < tcount) L.lists.kx[lk[u]] = __float_as_uint(kn[u]);
      }
    }

    float M1[2] = {FLT_MAX, FLT_MAX}, M2[2] = {FLT_MAX, FLT_MAX};
    int B1[2] = {0, 0};
    for (int blk = 0; blk < nblk; ++blk) {
      // lanes h = 1 read the same split row; their B operand is zero
      const u32x4 an = *(const u32x4*)(Ns + (blk * 32 + q) * 8);
      u32x4 af[4];
#pragma unroll
      for (int s2 = 0; s2 < 4; ++s2) af[s2] = *(const u32x4*)(Rs + swz(blk * 32 + q, 4 * h + s2));
      f32x16 acc[2];
#pragma unroll
      for (int u = 0; u < 2; ++u)
        acc[u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, an),
                                                         __builtin_bit_cast(bf16x8, ones), zero, 0, 0, 0);
#pragma unroll
      for (int s2 = 0; s2 < 4; ++s2)
#pragma unroll
        for (int u = 0; u < 2; ++u)
          acc[u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, af[s2]),
                                                           __builtin_bit_cast(bf16x8, kf[u][s2]), acc[u], 0, 0, 0);
#pragma unroll
      for (int u = 0; u < 2; ++u) reduce_block(acc[u], blk, M1[u], M2[u], B1[u]);
    }
    // lanes h = 0 decide the keys of tile tt, lanes h = 1 those of tile tt + 1
    decide_pair<FIRST>(M1[0], M2[0], B1[0], M1[1], M2[1], B1[1], h ? kn[1] : kn[0], h ? old[1] : old[0],
                       h ? lk[1] : lk[0], tt + h < tcount, h ? valid[1] : valid[0], N, cf, L.lists, wv, wn, un);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
#pragma unroll
      for (int s2 = 0; s2 < 4; ++s2) kf[u][s2] = kf_n[u][s2];
      kn[u] = kn_n[u];
      old[u] = old_n[u];
    }
  }
  if (lane == 0) {
    cnt.wcnt[wv] = wn;
    cnt.ucnt[wv] = un;
  }
  assign_epilogue<FIRST, false, 1>(Kbh, key0, tpw, Rs, nrm64 + bh * N, n, N, belong_bh, knorm + bh * n, mcount + bh,
                                   mrec + bh * n, kd[wave], L.lists);
}

// Key fragments of tile `tile` of a slice, and in later rounds the keys' |k|
// bound and previous group.  Keys outside 0 .. n - 1 read the nearest key
// instead (their results are never stored), so every lane loads
// unconditionally.
template <bool FIRST>
__device__ __forceinline__ void load_keys(const uint16_t* __restrict__ Kbh, const float* __restrict__ knorm_bh,
                                          const int32_t* __restrict__ belong_bh, int64_t tile, int n, int q, int h,
                                          u32x4 (&f)[4], float& knv, int& oldv) {
  const int64_t key = max((int64_t)0, min(tile * 32 + q, (int64_t)n - 1));
  const uint16_t* krow = Kbh + key * 64 + h * 32;
#pragma unroll
  for (int s2 = 0; s2 < 4; ++s2) f[s2] = *(const u32x4*)(krow + s2 * 8);
  if (!FIRST) {
    knv = knorm_bh[key];
    oldv = belong_bh[key];
  }
}

// k_assign_reg: the variant for N <= 32 NB (NB = 1..4).  Each lane keeps its
// A fragments of -2R and of the |r|^2 split for all NB blocks in VGPRs (read
// once from LDS), so the scoring loop issues no LDS reads; only the exact
// re-decisions read the LDS copy.  The key fragments of the next tile are
// loaded while the current one is scored (two register sets used in turn, no
// copies; the last tile's prefetch repeats it).  Same grid, LDS layout,
// scores, certification and outputs as k_assign_bf16.  FUSED (first round
// only): the workgroup also forms its partition sums of the round's centroid
// update (partition_sums), at most kFusedP per slice.
template <bool FIRST, int NB, bool FUSED>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_assign_reg(
    const uint16_t* __restrict__ K, const uint16_t* R, const uint16_t* nsplit, const double* nrm64,
    float* __restrict__ knorm, int32_t* __restrict__ belong, int32_t* __restrict__ mcount,
    unsigned long long* __restrict__ mrec, int n, int N, int tpw, float cm, float cp, FusedUpdate fu) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ double red[4];
  __shared__ AssignCounts cnt;
  __shared__ __align__(16) double kd[4][kExactB * 64];  // fp64 rows of queued keys, per wave
  constexpr int Npad = NB * 32;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5, q = lane & 31;
  const int64_t bh = blockIdx.y;
  if (tid == 0) cnt.nx = 0;
  const AssignLds L = assign_lds_layout(smem, Npad, tpw, FUSED, &cnt);
  const int64_t key0 = (int64_t)blockIdx.x * 4 * tpw * 32;
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const int64_t tile0 = key0 / 32 + (int64_t)wv * tpw;
  const int64_t ntiles = ((int64_t)n + 31) / 32;
  const int tcount = (int)max((int64_t)0, min((int64_t)tpw, ntiles - tile0));
  const uint16_t* Kbh = K + bh * (int64_t)n * 64;
  const float* knorm_bh = knorm + bh * n;
  const int32_t* belong_bh = belong + bh * n;
  // The first key tile (see the loop below) loads while the workgroup stages R.
  u32x4 kb[2][4];
  float knb[2] = {0.f, 0.f};
  int oldb[2] = {0, 0};
  load_keys<FIRST>(Kbh, knorm_bh, belong_bh, tile0 + min(0, tcount - 1), n, q, h, kb[0], knb[0], oldb[0]);
  // FUSED (first round): the initial representatives from the keys or the
  // given init; workgroup 0 of the slice writes C and clears the moved-key
  // counters of the next rounds
  __shared__ double nrm_l[FUSED ? Npad : 1];
  if (FUSED && blockIdx.x == 0 && tid == 0) {
    mcount[bh] = 0;
    mcount[gridDim.y + bh] = 0;
  }
  const double nmax =
      FUSED ? stage_init<Npad>(Kbh, fu.init ? fu.init + bh * (int64_t)N * 64 : nullptr, n, N,
                               blockIdx.x == 0 ? fu.C + bh * (int64_t)N * 64 : nullptr, L.Rs, L.Ns, nrm_l, red)
            : stage_reps<Npad>(R + bh * (int64_t)N * 64, nsplit + bh * N * 8, nrm64 + bh * N, N, Npad, L.Rs, L.Ns,
                               red);
  const double* nrm_x = FUSED ? (const double*)nrm_l : nrm64 + bh * N;  // |r|^2 for the exact decisions
  const float nmaxf = (float)nmax * (1.0f + 0x1p-20f);
  const float rmaxf = sqrtf(nmaxf) * (1.0f + 0x1p-20f);
  const Certify cf = {nmaxf, rmaxf, cm, cp};

  u32x4 af[NB][4], an[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    an[b] = *(const u32x4*)(L.Ns + (b * 32 + q) * 8);  // lanes h = 1 read it too; their B is zero
#pragma unroll
    for (int s2 = 0; s2 < 4; ++s2) af[b][s2] = *(const u32x4*)(L.Rs + swz(b * 32 + q, 4 * h + s2));
  }
  const u32x4 ones = h == 0 ? u32x4{0x3f803f80u, 0x3f80u, 0u, 0u} : u32x4{0u, 0u, 0u, 0u};
  // later rounds: the |r|^2 parts of the scores once for all tiles (the first
  // round, which holds more state, adds them per tile)
  constexpr bool kHoist = !FIRST;
  f32x16 nacc[NB];
  if (kHoist) norm_terms<NB>(an, ones, nacc);

  int wn = 0, un = 0;  // this wave's moved / uncertain entries (wave-uniform)
  auto score = [&](const u32x4 (&kf)[4], float& knv, int t, float& M1, float& M2, int& B1)
                   __attribute__((always_inline)) {
    if (FIRST) {
      knv = key_norm_bound(kf);
      L.lists.kx[(wv * tpw + t) * 32 + q] = __float_as_uint(knv);
    }
    score_tile<NB, kHoist>(af, an, ones, nacc, kf, M1, M2, B1);
  };
  // Two register sets used in turn: tile t + 1 is loaded while tile t is
  // scored (deeper rings measured no faster: the loop is bound by the
  // scoring, not by the loads); loads past the last tile repeat it.  The
  // tiles are decided in pairs (decide_pair).  The scheduling barriers keep
  // each prefetch ahead of the tile it overlaps.
  for (int t = 0; t < tcount; t += 2) {
    float M1a, M2a, M1b, M2b;
    int B1a, B1b;
    load_keys<FIRST>(Kbh, knorm_bh, belong_bh, tile0 + min(t + 1, tcount - 1), n, q, h, kb[1], knb[1], oldb[1]);
    __builtin_amdgcn_sched_barrier(0);
    score(kb[0], knb[0], t, M1a, M2a, B1a);
    const float kna = knb[0];
    const int olda = oldb[0];
    load_keys<FIRST>(Kbh, knorm_bh, belong_bh, tile0 + min(t + 2, tcount - 1), n, q, h, kb[0], knb[0], oldb[0]);
    __builtin_amdgcn_sched_barrier(0);
    score(kb[1], knb[1], min(t + 1, tcount - 1), M1b, M2b, B1b);  // past the last tile: a repeat, not staged
    // lanes h = 0 decide the keys of tile t, lanes h = 1 those of tile t + 1
    const int lk = (wv * tpw + t + h) * 32 + q;
    const bool stage = t + h < tcount;
    decide_pair<FIRST>(M1a, M2a, B1a, M1b, M2b, B1b, h ? knb[1] : kna, h ? oldb[1] : olda, lk, stage,
                       stage && key0 + lk < n, N, cf, L.lists, wv, wn, un);
  }
  if (lane == 0) {
    cnt.wcnt[wv] = wn;
    cnt.ucnt[wv] = un;
  }
  assign_epilogue<FIRST, FUSED, kExactB>(Kbh, key0, tpw, L.Rs, nrm_x, n, N, belong + bh * n, knorm + bh * n,
                                          mcount + bh, mrec + bh * n, kd[wave], L.lists);
  if (FUSED) {
    __shared__ PartLds pl;
    const int nk = (int)min((int64_t)4 * tpw * 32, (int64_t)n - key0);
    static_assert(FIRST || !FUSED, "partition sums are formed in the first round only");
    partition_sums(Kbh, key0, nk, N, L.lists, (uint32_t*)smem, fused_words(Npad, 4 * tpw * 32), pl, fu);
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
                                                double* __restrict__ nrm64, uint16_t* __restrict__ nsplit) {
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
    finalize_rep<S>(c, row, R, nrm64, nsplit);
  } else {
    out[row * 64 + lane] = (float)acc;
  }
}

// ------------------------------------------------------------------ group sums (bf16)
// run_sums: the rows of a group-sorted entry list (ent: key | leave << 31;
// eg: the entry's group within the workgroup's block) added into the LDS sums
// acc[g][64] by one workgroup of 4 waves.  The list is cut into 32 contiguous
// ranges, one per 8-lane slot (lane j of a slot holds features 8 j .. 8 j + 7
// of the slot's row, one 16-byte load); a slot adds its rows in fp64
// registers while the group stays the same and adds the partial sum into acc
// with LDS atomics when it changes, so the atomics scale with the groups, not
// the rows.  The member sums are exact in fp64 (see the bf16 member sums
// above), so neither the cut nor the order of the atomics can change a bit.
constexpr int kRunU = 8;  // rows per slot and batch (two batches in flight)
__device__ __forceinline__ void run_sums(const uint32_t* ent, const uint8_t* eg, int ne,
                                         const uint16_t* __restrict__ Xb, double* acc, int wave, int lane) {
  if (ne <= 0) return;
  const int j = lane & 7, gsl = 8 * wave + (lane >> 3);
  const int b0 = (int)((int64_t)gsl * ne / 32), b1 = (int)((int64_t)(gsl + 1) * ne / 32);
  const int steps = (ne + 31) / 32;  // >= every slot's range (they differ by at most one)
  double a[8] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
  int cur = -1;
  auto load = [&](int k0, uint32_t (&ei)[kRunU], int (&gi)[kRunU], u32x4 (&w)[kRunU]) {
#pragma unroll
    for (int u = 0; u < kRunU; ++u) {
      const int e = min(b0 + k0 + u, ne - 1);
      ei[u] = ent[e];
      gi[u] = eg[e];
      w[u] = *(const u32x4*)(Xb + (int64_t)(ei[u] & 0x7fffffffu) * 64 + 8 * j);
    }
  };
  auto flush = [&]() {
    double* p = acc + cur * 64 + 8 * j;
#pragma unroll
    for (int f = 0; f < 8; ++f) {
      atomicAdd(p + f, a[f]);
      a[f] = 0.0;
    }
  };
  auto add = [&](int k0, const uint32_t (&ei)[kRunU], const int (&gi)[kRunU], const u32x4 (&w)[kRunU]) {
#pragma unroll
    for (int u = 0; u < kRunU; ++u) {
      if (b0 + k0 + u >= b1) break;
      if (gi[u] != cur) {
        if (cur >= 0) flush();
        cur = gi[u];
      }
      const double sg = (ei[u] >> 31) ? -1.0 : 1.0;
#pragma unroll
      for (int f = 0; f < 8; ++f)
        a[f] = fma(sg, (double)bf16_to_f32((w[u][f >> 1] >> (16 * (f & 1))) & 0xffffu), a[f]);
    }
  };
  uint32_t eA[kRunU], eB[kRunU];
  int gA[kRunU], gB[kRunU];
  u32x4 wA[kRunU], wB[kRunU];
  load(0, eA, gA, wA);
  for (int k0 = 0; k0 < steps; k0 += 2 * kRunU) {
    if (k0 + kRunU < steps) load(k0 + kRunU, eB, gB, wB);
    add(k0, eA, gA, wA);
    if (k0 + kRunU >= steps) break;
    if (k0 + 2 * kRunU < steps) load(k0 + 2 * kRunU, eA, gA, wA);
    add(k0 + kRunU, eB, gB, wB);
  }
  if (cur >= 0) flush();
}

// The member sums of the bf16 path are exact in fp64 (see above), so they can
// be accumulated in any order and split any way: no global bucketing.
//
// k_gsum: grid (ceil(N / 32), BH), 256 threads.  Workgroup x owns groups
// g0 = 32 x .. g0 + 31 of slice bh and finishes them itself:
//   MODE 0 (first round): S = sum of the member key rows, count = members
//   MODE 2 (value sums):  vsum = (float) sum of the member value rows
//   MODE 3 (value sums for the attention): the bf16 value means, transposed,
//           and the log2(count) score bias, as k_attend_prep forms them
// MODE 0 then sets C = (float)(S / count) (an empty group keeps C), R =
// bf16(C), the canonical fp64 |r|^2 (fma chain over c = 0..63, one lane per
// group) and its split.  (The later rounds' update is k_gdelta.)
//
// Per chunk of keys, all loaded at once:
// 1. count the keys of every owned group and scatter them into an LDS list
//    sorted by group (a local counting sort; one LDS atomic per key);
// 2. run_sums adds the rows into the LDS sums;
// 3. finish the owned groups.
constexpr int kGsumG = 32;
constexpr int kGsumList = 8192;  // entry capacity of the sorted chunk list
template <int MODE>
__global__ __launch_bounds__(256) void k_gsum(const uint16_t* __restrict__ X, const int32_t* __restrict__ belong,
                                              int n, int N, double* __restrict__ S64,
                                              int32_t* __restrict__ count, float* __restrict__ out, uint16_t* __restrict__ R,
                                              double* __restrict__ nrm64, uint16_t* __restrict__ nsplit,
                                              float inv_sl2e, int vts) {
  __shared__ uint32_t ent[kGsumList];  // keys sorted by group
  __shared__ uint8_t eg[kGsumList];    // their groups, relative to g0
  __shared__ double acc[kGsumG * 64];  // [g][c] sums of this workgroup's groups
  __shared__ int ecnt[kGsumG], eoff[kGsumG + 1], ecur[kGsumG], dcnt[kGsumG];
  float* rsh = (float*)ent;            // [32][65] bf16 representatives, after the sums
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t bh = blockIdx.y;
  const int g0 = blockIdx.x * kGsumG, ng = min(kGsumG, N - g0);
  for (int i = tid; i < kGsumG * 64; i += 256) acc[i] = 0.0;
  if (tid < kGsumG) dcnt[tid] = 0;

  const int64_t total = n;
  constexpr int CH = kGsumList;  // keys per chunk
  constexpr int PER = CH / 256;
  const uint16_t* Xb = X + bh * (int64_t)n * 64;
  for (int64_t c0 = 0; c0 < total; c0 += CH) {
    int kv[PER], gj[PER];
    // every lane loads (index clamped into the chunk) so that the loads overlap
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int64_t e = c0 + tid + 256 * u, ec = min(e, total - 1);
      kv[u] = (int)e;
      gj[u] = belong[bh * n + ec] - g0;
    }
#pragma unroll
    for (int u = 0; u < PER; ++u)
      if (c0 + tid + 256 * u >= total) gj[u] = -1;
    if (tid < kGsumG) ecnt[tid] = 0;
    __syncthreads();
    // 1. count, lay out, scatter
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int g = gj[u];
      if ((unsigned)g < (unsigned)ng) {
        atomicAdd(&ecnt[g], 1);
        if (MODE == 0) atomicAdd(&dcnt[g], 1);
      }
    }
    __syncthreads();
    if (wave == 0) {
      const int c = lane < kGsumG ? ecnt[lane] : 0;
      int incl = c;  // inclusive scan over the 32 groups
#pragma unroll
      for (int off = 1; off < 32; off <<= 1) {
        const int y = __shfl_up(incl, off);
        if (lane >= off) incl += y;
      }
      if (lane < kGsumG) {
        eoff[lane] = incl - c;
        ecur[lane] = incl - c;
      }
      if (lane == kGsumG - 1) eoff[kGsumG] = incl;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int g = gj[u];
      if ((unsigned)g < (unsigned)ng) {
        const int pos = atomicAdd(&ecur[g], 1);
        ent[pos] = (uint32_t)kv[u];
        eg[pos] = (uint8_t)g;
      }
    }
    __syncthreads();
    // 2. the rows, summed per group
    run_sums(ent, eg, eoff[kGsumG], Xb, acc, wave, lane);
    __syncthreads();
  }

  // 3. finish the owned groups: element (g, c) = (idx / 64, idx % 64), 8 per thread
  constexpr int EPT = kGsumG * 64 / 256;
  int pc[EPT];
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    const int idx = tid + 256 * u, g = idx >> 6;
    const int64_t row = bh * N + g0 + min(g, ng - 1);
    pc[u] = MODE == 3 ? count[row] : 0;
  }
  __syncthreads();  // (total == 0: dcnt, acc initialised above)
  if (MODE == 3) {
    // value means mu = (float) sum / count (0 for an empty or padded group)
    // as bf16, transposed through LDS into Vt[feature][group] (R, 8-byte
    // segments), and the score bias log2(count) / sl2e (-inf if empty) into
    // out[bh][Npad]
    uint16_t* mt = (uint16_t*)ent;  // [64][36]
#pragma unroll
    for (int u = 0; u < EPT; ++u) {
      const int idx = tid + 256 * u, g = idx >> 6, c = idx & 63;
      const float vs = g < ng ? (float)acc[g * 64 + c] : 0.f;
      const int cnt = g < ng ? pc[u] : 0;
      mt[c * 36 + g] = (uint16_t)f32_to_bf16(cnt > 0 ? vs / (float)cnt : 0.f);
      if (c == 0) out[bh * ((N + 31) & ~31) + g0 + g] = cnt > 0 ? log2f((float)cnt) * inv_sl2e : -INFINITY;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int x = tid + 256 * u, f = x >> 3, q4 = x & 7;  // 64 features x 8 segments of 4 groups
      *(uint2*)(R + (bh * 64 + f) * (int64_t)vts + g0 + 4 * q4) = *(const uint2*)(mt + f * 36 + 4 * q4);
    }
    return;
  }
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    const int idx = tid + 256 * u, g = idx >> 6, c = idx & 63;
    if (g >= ng) continue;
    const int64_t row = bh * N + g0 + g;
    const double s = acc[g * 64 + c];
    if (MODE == 2) {
      out[row * 64 + c] = (float)s;
      continue;
    }
    const double S = s;
    const int cnt = dcnt[g];
    S64[row * 64 + c] = S;
    if (c == 0) count[row] = cnt;
    float cf;
    if (cnt > 0) {
      cf = (float)(S / (double)cnt);
      out[row * 64 + c] = cf;
    } else {
      cf = out[row * 64 + c];
    }
    const float r = BF16::rep(cf);
    BF16::store(R, row * 64 + c, r);
    rsh[g * 65 + c] = r;
  }
  if (MODE == 2) return;
  __syncthreads();
  if (tid < ng) {
    const int64_t row = bh * N + g0 + tid;
    double nrm = 0.0;
#pragma unroll 8
    for (int c = 0; c < 64; ++c) {
      const double rc = (double)rsh[tid * 65 + c];
      nrm = fma(rc, rc, nrm);
    }
    nrm64[row] = nrm;
    write_nsplit(nrm, nsplit + row * 8);
  }
}

// ------------------------------------------------------------------ later-round update (bf16)
// k_gdelta: grid (ceil(N / 32), BH), 256 threads: the later rounds' update
// of workgroup x's groups g0 = 32 x .. g0 + 31 of slice bh from the round's
// moved-key records (key, group joined, group left): S += joins - leaves,
// count += joins - leaves, then C, R, |r|^2 and its split as k_gsum forms them
// for the groups any record touches.  In the later rounds few keys move, so
// the update is mostly latency:
//   - the owned groups' previous sums and counts are requested first, so
//     that their loads overlap the record pass;
//   - the touched (key, side) entries are sorted by group in LDS (counting
//     sort, no padding);
//   - run_sums adds the rows (joins +, leaves -).
constexpr int kDeltaCh = 4096;  // records per pass (at most 2 entries each)
__global__ __launch_bounds__(256) void k_gdelta(const uint16_t* __restrict__ X,
                                                const unsigned long long* __restrict__ mrec,
                                                const int32_t* __restrict__ mcount_cur,
                                                int32_t* __restrict__ mcount_next, int n, int N,
                                                double* __restrict__ S64, int32_t* __restrict__ count,
                                                float* __restrict__ C, uint16_t* __restrict__ R,
                                                double* __restrict__ nrm64, uint16_t* __restrict__ nsplit) {
  __shared__ uint32_t ent[2 * kDeltaCh];  // key | leave << 31, sorted by group
  __shared__ uint8_t eg[2 * kDeltaCh];    // its group, relative to g0
  __shared__ double acc[kGsumG * 64];
  __shared__ float rsh[kGsumG * 65];
  __shared__ int ecnt[kGsumG], ecur[kGsumG], eoff[kGsumG + 1], dcnt[kGsumG], hit[kGsumG];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t bh = blockIdx.y;
  const int g0 = blockIdx.x * kGsumG, ng = min(kGsumG, N - g0);

  // previous sums and counts: element (g, c) = (idx / 64, idx % 64), 8 per thread
  constexpr int EPT = kGsumG * 64 / 256;
  double prev[EPT];
  int pc[EPT];
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    const int idx = tid + 256 * u, g = idx >> 6, c = idx & 63;
    const int64_t row = bh * N + g0 + min(g, ng - 1);
    prev[u] = S64[row * 64 + c];
    pc[u] = count[row];
  }
  for (int i = tid; i < kGsumG * 64; i += 256) acc[i] = 0.0;
  if (tid < kGsumG) {
    ecnt[tid] = 0;
    dcnt[tid] = 0;
    hit[tid] = 0;
  }

  // (a slice records at most n moved keys; the clamp keeps the loads below in
  // bounds even if the workspace was corrupted, e.g. shared by overlapping calls)
  const int64_t total = min((int64_t)mcount_cur[bh], (int64_t)n);
  constexpr int PER = kDeltaCh / 256;
  const uint16_t* Xb = X + bh * (int64_t)n * 64;
  for (int64_t c0 = 0; c0 < total; c0 += kDeltaCh) {
    uint32_t kv[PER];
    int gj[PER], gl[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int64_t e = c0 + tid + 256 * u, ec = min(e, total - 1);
      const unsigned long long r = mrec[bh * n + ec];
      kv[u] = (uint32_t)min((int)(r >> 32) & 0x7fffffff, n - 1);
      gj[u] = e < total ? (int)(r & 0xffffu) - g0 : -1;
      gl[u] = e < total ? (int)((r >> 16) & 0xffffu) - g0 : -1;
    }
    __syncthreads();  // zeroed counters; the previous pass is done with the list
    // 1. count, offsets, scatter (the list keeps the groups in order)
#pragma unroll
    for (int u = 0; u < PER; ++u)
#pragma unroll
      for (int side = 0; side < 2; ++side) {
        const int g = side ? gl[u] : gj[u];
        if ((unsigned)g < (unsigned)ng) {
          atomicAdd(&ecnt[g], 1);
          atomicAdd(&dcnt[g], side ? -1 : 1);
          hit[g] = 1;
        }
      }
    __syncthreads();
    if (wave == 0) {
      const int c = lane < kGsumG ? ecnt[lane] : 0;
      int incl = c;
#pragma unroll
      for (int off = 1; off < 32; off <<= 1) {
        const int y = __shfl_up(incl, off);
        if (lane >= off) incl += y;
      }
      if (lane < kGsumG) {
        eoff[lane] = incl - c;
        ecur[lane] = incl - c;
      }
      if (lane == kGsumG - 1) eoff[kGsumG] = incl;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < PER; ++u)
#pragma unroll
      for (int side = 0; side < 2; ++side) {
        const int g = side ? gl[u] : gj[u];
        if ((unsigned)g < (unsigned)ng) {
          const int pos = atomicAdd(&ecur[g], 1);
          ent[pos] = kv[u] | ((uint32_t)side << 31);
          eg[pos] = (uint8_t)g;
        }
      }
    __syncthreads();
    // 2. the rows, summed per group
    run_sums(ent, eg, eoff[kGsumG], Xb, acc, wave, lane);
    __syncthreads();
    if (tid < kGsumG) ecnt[tid] = 0;
  }
  __syncthreads();

  // the touched groups: S, count, C (an empty group keeps C), R, |r|^2
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    const int idx = tid + 256 * u, g = idx >> 6, c = idx & 63;
    if (g >= ng || !hit[g]) continue;
    const int64_t row = bh * N + g0 + g;
    const double S = prev[u] + acc[g * 64 + c];
    const int cnt = pc[u] + dcnt[g];
    S64[row * 64 + c] = S;
    if (c == 0) count[row] = cnt;
    float cf;
    if (cnt > 0) {
      cf = (float)(S / (double)cnt);
      C[row * 64 + c] = cf;
    } else {
      cf = C[row * 64 + c];
    }
    const float r = BF16::rep(cf);
    BF16::store(R, row * 64 + c, r);
    rsh[g * 65 + c] = r;
  }
  __syncthreads();
  if (tid < ng && hit[tid]) {
    const int64_t row = bh * N + g0 + tid;
    double nrm = 0.0;
#pragma unroll 8
    for (int c = 0; c < 64; ++c) {
      const double rc = (double)rsh[tid * 65 + c];
      nrm = fma(rc, rc, nrm);
    }
    nrm64[row] = nrm;
    write_nsplit(nrm, nsplit + row * 8);
  }
  if (blockIdx.x == 0 && tid == 0) mcount_next[bh] = 0;
}

// ------------------------------------------------------------------ attention (bf16)
// grid (ceil(Npad/64), BH), 256 threads; groups g0 = 64 x .. (padded groups
// past N get zeros).  Each wave reads 16 groups' rows (lane = feature), the
// transposed value means go through LDS and out as whole row segments.
// Vt holds the group's value MEAN vsum_j / count_j (bf16) so that the count
// weight can move into the exponent: o_i = sum_j c_j e_ij mu_j / sum_j c_j e_ij
// with c_j e_ij = exp2(t_ij + log2 c_j).  ginit_j = log2(c_j) / sl2e is added to
// the score accumulator (-inf for an empty group, which drops it).
__global__ __launch_bounds__(256) void k_attend_prep(const float* __restrict__ centroid,
                                                     const int32_t* __restrict__ count,
                                                     const float* __restrict__ vsum, float inv_sl2e,
                                                     int N, int vts, uint16_t* __restrict__ Rq,
                                                     uint16_t* __restrict__ Vt, float* __restrict__ ginit) {
  __shared__ uint16_t mt[64][66];  // [feature][group] value means, bf16
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t bh = blockIdx.y;
  const int Npad = (N + 31) & ~31;
  const int g0 = blockIdx.x * 64, ng = min(64, Npad - g0);
  int cnt[16];
  float vs[16], cen[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int g = g0 + wave * 16 + i;
    const int64_t row = bh * N + min(g, N - 1);
    cnt[i] = g < N ? count[row] : 0;
    vs[i] = vsum[row * 64 + lane];
    if (Rq) cen[i] = centroid[row * 64 + lane];
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int gl = wave * 16 + i, g = g0 + gl;
    if (gl >= ng) break;
    const int64_t row = bh * N + g;
    if (Rq && g < N) Rq[row * 64 + lane] = (uint16_t)f32_to_bf16(cen[i]);
    const float mu = cnt[i] > 0 ? vs[i] / (float)cnt[i] : 0.f;
    mt[lane][gl] = (uint16_t)f32_to_bf16(mu);
    if (lane == 0) ginit[bh * Npad + g] = cnt[i] > 0 ? log2f((float)cnt[i]) * inv_sl2e : -INFINITY;
  }
  __syncthreads();
  const int np = ng / 2;  // group pairs per feature row
  for (int idx = tid; idx < 64 * np; idx += 256) {
    const int f = idx / np, pr = idx % np;
    *(uint32_t*)(Vt + (bh * 64 + f) * vts + g0 + 2 * pr) = *(const uint32_t*)&mt[f][2 * pr];
  }
}

// grid (ceil(tiles / (4 * tpw)), BH), 256 threads, N <= 32 NB (NB <= 8).
// LDS: sign(scale) R as [Npad][kRs] bf16, Vt as [64][vts] bf16, ginit [Npad],
// one [32][kOs] bf16 tile per wave (the wave's query tile, then its output
// tile, both moved between HBM and LDS as whole rows).  Each wave owns tpw
// consecutive 32-query tiles; the next tile's queries are
// loaded while the current one is processed (two register sets in turn).
// Scores: MFMA with A = R rows (32 groups), B = Q tile (32 queries);
// accumulator init ginit; t = acc * sl2e.  N <= 128: all scores of the tile,
// then the exact max over its groups.  N > 128: online max per 32-group
// block, rescaled only when the block max exceeds the running max by more than
// 8 (log2 units).  Combine: MFMA with A = Vt rows (32 features x 16 groups), B =
// bf16(exp2(t - m)) taken straight from the score registers (the group order
// of the contraction axis is the score layout's, applied identically to A).
// The denominator sum_j c_j e_ij comes from the matrix core too: a third
// combine tile whose A operand is a constant row of ones (row 0) adds the same
// bf16 weights the numerator uses.
// Queries past n are computed as the slice's last query and store that
// query's (identical) output, so every lane loads and stores unconditionally.
template <int NB>
__global__ __launch_bounds__(256) void k_attend_bf16(const uint16_t* __restrict__ Q,
                                                     const uint16_t* __restrict__ R,
                                                     const uint16_t* __restrict__ Vt,
                                                     const float* __restrict__ ginit, int n, int N,
                                                     int vts, float sl2e, uint32_t rsign, int tpw,
                                                     uint16_t* __restrict__ O) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int Npad = NB * 32;
  uint16_t* Rs = (uint16_t*)smem;
  uint16_t* Vs = Rs + Npad * kRs;
  float* gi = (float*)(Vs + 64 * vts);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5, q = lane & 31;
  uint16_t* Ow = (uint16_t*)(gi + Npad) + wave * 32 * kOs;  // this wave's output tile
  const int64_t bh = blockIdx.y;
  const int64_t tile0 = ((int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(wave)) * tpw;
  const int64_t ntiles = ((int64_t)n + 31) / 32;
  const int tcount = (int)max((int64_t)0, min((int64_t)tpw, ntiles - tile0));
  const uint16_t* Qbh = Q + bh * (int64_t)n * 64;
  uint16_t* Obh = O + bh * (int64_t)n * 64;
  // Query tile t in row-major order: lane l holds 16 bytes (chunk l % 8) of
  // rows l / 8 + 8 k, so each load instruction reads 8 whole 128-byte rows.
  auto qload = [&](int t, u32x4 (&qc)[4]) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int64_t qi = min((tile0 + t) * 32 + 8 * k + (lane >> 3), (int64_t)n - 1);
      qc[k] = *(const u32x4*)(Qbh + qi * 64 + (lane & 7) * 8);
    }
  };
  // The first query tiles (see the ring below) load while the workgroup
  // stages R, the value means and the bias; every staging load is issued
  // (rows clamped into the slice) before any of them is stored.
  constexpr int D = kAttDepth;
  u32x4 qb[D + 1][4];
#pragma unroll
  for (int r = 0; r < D; ++r) qload(min(r, max(tcount - 1, 0)), qb[r]);
  const uint16_t* Rbh = R + bh * (int64_t)N * 64;
  const uint16_t* Vbh = Vt + bh * 64 * (int64_t)vts;
  constexpr int RIT = Npad * 8 / 256, VIT = 64 * (Npad / 4) / 256;
  u32x4 rv[RIT];
  u32x2 vv[VIT];
#pragma unroll
  for (int it = 0; it < RIT; ++it) {
    const int idx = tid + 256 * it, row = idx >> 3, ch = idx & 7;
    rv[it] = *(const u32x4*)(Rbh + (int64_t)min(row, N - 1) * 64 + ch * 8);
  }
  // rows of Vt are 8-byte aligned (vts = 128k + 4 keeps the combine's LDS reads conflict-free)
#pragma unroll
  for (int it = 0; it < VIT; ++it) {
    const int idx = tid + 256 * it, row = idx / (Npad / 4), ch = idx % (Npad / 4);
    vv[it] = *(const u32x2*)(Vbh + (int64_t)row * vts + ch * 4);
  }
  const float gx = tid < Npad ? ginit[bh * Npad + tid] : -INFINITY;
#pragma unroll
  for (int it = 0; it < RIT; ++it) {
    const int idx = tid + 256 * it, row = idx >> 3, ch = idx & 7;
    const u32x4 v = row < N ? rv[it] ^ u32x4{rsign, rsign, rsign, rsign} : u32x4{0u, 0u, 0u, 0u};
    *(u32x4*)(Rs + row * kRs + ch * 8) = v;
  }
#pragma unroll
  for (int it = 0; it < VIT; ++it) {
    const int idx = tid + 256 * it, row = idx / (Npad / 4), ch = idx % (Npad / 4);
    *(u32x2*)(Vs + row * vts + ch * 4) = vv[it];
  }
  if (tid < Npad) gi[tid] = gx;
  const int any = __syncthreads_or(gx != -INFINITY);

  // A operand of the denominator tile: row 0 (lane 0 and its h = 1 partner) all ones
  const u32x4 ones_row = q == 0 ? u32x4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u} : u32x4{0u, 0u, 0u, 0u};

  auto run = [&](int t, const u32x4 (&qc)[4]) __attribute__((always_inline)) {
    // to MFMA B fragments through the wave's LDS tile: lane (h, q) takes
    // features 32 h + 8 s .. +7 of query q at k-step s
#pragma unroll
    for (int k = 0; k < 4; ++k) *(u32x4*)(Ow + (8 * k + (lane >> 3)) * kOs + (lane & 7) * 8) = qc[k];
    u32x4 qf[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) qf[s] = *(const u32x4*)(Ow + q * kOs + h * 32 + s * 8);
    f32x16 o0, o1, o2;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      o0[v] = 0.f;
      o1[v] = 0.f;
      o2[v] = 0.f;
    }
    float mt = -INFINITY;
    if (NB <= 4 && any) {
      // All scores first (NB accumulators), then one exact max over every
      // group of the tile, then exp2 / pack / combine per block: no branch
      // inside the tile, so one block's MFMAs overlap another's VALU work.
      f32x16 acc[NB];
#pragma unroll
      for (int blk = 0; blk < NB; ++blk) {
        const float* gb = gi + blk * 32 + 4 * h;
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[blk][v] = gb[8 * (v >> 2) + (v & 3)];
        const uint16_t* ar = Rs + (blk * 32 + q) * kRs + h * 32;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const u32x4 a = *(const u32x4*)(ar + s * 8);
          acc[blk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                             __builtin_bit_cast(bf16x8, qf[s]), acc[blk], 0, 0, 0);
        }
      }
      float bm = -INFINITY;
#pragma unroll
      for (int blk = 0; blk < NB; ++blk)
#pragma unroll
        for (int v = 0; v < 16; ++v) bm = __builtin_amdgcn_fmed3f(bm, acc[blk][v], INFINITY);
      {
        const u32x2 p = halves(__float_as_uint(bm));
        bm = __builtin_amdgcn_fmed3f(__uint_as_float(p[0]), __uint_as_float(p[1]), INFINITY);
      }
      // some group is non-empty (any), so bm is finite; empty groups give exp2(-inf) = 0
      const float nm = -bm * sl2e;
#pragma unroll
      for (int blk = 0; blk < NB; ++blk) {
        u32x4 b0, b1;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          b0[w] = pack_bf16x2(__builtin_amdgcn_exp2f(fmaf(acc[blk][2 * w], sl2e, nm)),
                              __builtin_amdgcn_exp2f(fmaf(acc[blk][2 * w + 1], sl2e, nm)));
          b1[w] = pack_bf16x2(__builtin_amdgcn_exp2f(fmaf(acc[blk][8 + 2 * w], sl2e, nm)),
                              __builtin_amdgcn_exp2f(fmaf(acc[blk][8 + 2 * w + 1], sl2e, nm)));
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
          o2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, ones_row),
                                                       __builtin_bit_cast(bf16x8, bsp), o2, 0, 0, 0);
        }
      }
    } else if (any) {
#pragma unroll
      for (int blk = 0; blk < NB; ++blk) {
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
        for (int v = 1; v < 16; ++v) bm = __builtin_amdgcn_fmed3f(bm, acc[v], INFINITY);
        {
          const u32x2 p = halves(__float_as_uint(bm));
          bm = __builtin_amdgcn_fmed3f(__uint_as_float(p[0]), __uint_as_float(p[1]), INFINITY);
        }
        if (bm == -INFINITY) continue;  // every group of this block is empty (uniform)
        const float bmt = bm * sl2e;
        if (mt == -INFINITY) {  // first non-empty block: nothing to rescale
          mt = bmt;
        } else if (bmt > mt + 8.0f) {
          const float alpha = __builtin_amdgcn_exp2f(mt - bmt);
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            o0[v] *= alpha;
            o1[v] *= alpha;
          }
          o2[0] *= alpha;
          mt = bmt;
        }
        float e[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) e[v] = __builtin_amdgcn_exp2f(fmaf(acc[v], sl2e, -mt));
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
          o2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, ones_row),
                                                       __builtin_bit_cast(bf16x8, bsp), o2, 0, 0, 0);
        }
      }
    }
    // row 0 of the third tile (register 0 of lanes h = 0) is the denominator of query q
    const float stot = __uint_as_float(halves(__float_as_uint(o2[0]))[0]);
    const float inv = any ? 1.0f / stot : 0.f;  // no group at all: zero output
    // The output tile goes through the wave's LDS tile (rows of kOs bf16) so
    // that each store instruction writes 8 whole 128-byte rows.
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const u32x2 w0 = {pack_bf16x2(o0[4 * r] * inv, o0[4 * r + 1] * inv),
                        pack_bf16x2(o0[4 * r + 2] * inv, o0[4 * r + 3] * inv)};
      const u32x2 w1 = {pack_bf16x2(o1[4 * r] * inv, o1[4 * r + 1] * inv),
                        pack_bf16x2(o1[4 * r + 2] * inv, o1[4 * r + 3] * inv)};
      *(u32x2*)(Ow + q * kOs + 8 * r + 4 * h) = w0;
      *(u32x2*)(Ow + q * kOs + 32 + 8 * r + 4 * h) = w1;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int row = 8 * k + (lane >> 3), ch = lane & 7;
      const u32x4 v = *(const u32x4*)(Ow + row * kOs + ch * 8);
      *(u32x4*)(Obh + min((tile0 + t) * 32 + row, (int64_t)n - 1) * 64 + ch * 8) = v;
    }
  };
  if (tcount <= 0) return;
  // Ring of kAttDepth + 1 register sets: tile t + kAttDepth is loaded while
  // tile t is processed.  Loads past the last tile repeat it.  The scheduling
  // barriers keep each prefetch ahead of the tile it overlaps.
  for (int t0 = 0; t0 < tcount; t0 += D + 1) {
#pragma unroll
    for (int r = 0; r <= D; ++r) {
      const int t = t0 + r;
      if (t >= tcount) break;
      qload(min(t + D, tcount - 1), qb[(r + D) % (D + 1)]);
      __builtin_amdgcn_sched_barrier(0);
      run(t, qb[r]);
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

constexpr size_t kAssignLdsMax = 160 * 1024 - 3 * 1024;  // dynamic LDS budget (static arrays use the rest)

size_t assign_lds(int N, int tpw = 12, bool fused = false) {  // see assign_lds_layout
  const int Npad = (N + 31) & ~31, cap4 = 4 * tpw * 32;
  return (size_t)assign_region_a(Npad, cap4, fused) + (size_t)3 * cap4 * 4;
}
size_t bucket_lds(int N) { return (size_t)16 * N * 8 + (size_t)2 * N * 4; }
size_t attend_lds(int N) {
  const int Npad = (N + 31) & ~31;
  return (size_t)Npad * kRs * 2 + (size_t)64 * vt_stride(N) * 2 + (size_t)Npad * 4 + (size_t)4 * 32 * kOs * 2;
}

// Raise the dynamic-LDS limit of the kernels that can exceed 64 KB to the
// most they ever request.  A failure here is not fatal (the launch reports any
// real problem), so the error it leaves behind is cleared.
void set_lds_limits() {
  static std::once_flag once;
  std::call_once(once, [] {
    (void)hipFuncSetAttribute((const void*)k_assign_bf16<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)kAssignLdsMax);
    (void)hipFuncSetAttribute((const void*)k_assign_bf16<false>, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)kAssignLdsMax);
    (void)hipFuncSetAttribute((const void*)k_bucket, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)bucket_lds(kMaxGroups));
    for (const void* f : {(const void*)k_attend_bf16<1>, (const void*)k_attend_bf16<2>, (const void*)k_attend_bf16<3>,
                          (const void*)k_attend_bf16<4>, (const void*)k_attend_bf16<5>, (const void*)k_attend_bf16<6>,
                          (const void*)k_attend_bf16<7>, (const void*)k_attend_bf16<8>})
      (void)hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)attend_lds(kAttMaxN));
    (void)hipGetLastError();
  });
}

inline unsigned cdiv(int64_t a, int64_t b) { return (unsigned)((a + b - 1) / b); }

// Workgroups of 256 threads that the current device holds at once for `fn`
// with `lds` bytes of dynamic LDS (runtime occupancy query, cached).
int64_t resident_wgs(const void* fn, size_t lds) {
  static std::mutex mu;
  static std::map<std::tuple<int, const void*, size_t>, int64_t> cache;
  int dev = 0;
  (void)hipGetDevice(&dev);
  std::lock_guard<std::mutex> lock(mu);
  const auto key = std::make_tuple(dev, fn, lds);
  const auto it = cache.find(key);
  if (it != cache.end()) return it->second;
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) cus = 1;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 256, lds) != hipSuccess || per_cu < 1) per_cu = 1;
  (void)hipGetLastError();
  return cache[key] = (int64_t)cus * per_cu;
}

// Tiles per wave so that a grid of (ceil(tiles / (4 tpw)), BH) workgroups of
// 4 waves fits in one round of `resident` workgroups (at least 1, at most cap).
int64_t tiles_per_wave(int64_t tiles, int64_t BH, int64_t resident, int64_t cap) {
  const int64_t per_slice = max((int64_t)1, resident / max((int64_t)1, BH));
  const int64_t tpw = (tiles + 4 * per_slice - 1) / (4 * per_slice);
  return tpw < 1 ? 1 : (tpw > cap ? cap : tpw);
}

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
  w.nsplit = (uint16_t*)take(BH * N * 16);
  w.knorm = (float*)take(BH * n * 4);
  w.belong = (int32_t*)take(BH * n * 4);
  w.perm = (int32_t*)take(BH * n * 4);
  w.goff = (int32_t*)take(BH * N * 4);
  w.count = (int32_t*)take(BH * N * 4);
  w.vsum = (float*)take(BH * N * 64 * 4);
  w.Rq = (uint16_t*)take(BH * N * 64 * 2);
  w.Vt = (uint16_t*)take(BH * 64 * (int64_t)vt_stride((int)N) * 2);
  w.ginit = (float*)take(BH * Npad * 4);
  w.S64 = (double*)take(BH * N * 64 * 8);
  w.mcount = (int32_t*)take(2 * BH * 4);
  w.mrec = (unsigned long long*)take(BH * n * 8);
  const int64_t fp = d.dtype == 1 && Npad <= kFusedG ? kFusedP : 0;  // fused-update partitions
  w.Sp = (double*)take(BH * fp * N * 64 * 8);
  w.cntp = (int32_t*)take(BH * fp * N * 4);
  w.pbits = (uint32_t*)take(BH * fp * 4 * 4);
  w.lxs = (double*)take(lloyd_exchange_rows(d) * 64 * 8);
  w.lxc = (int32_t*)take(lloyd_exchange_rows(d) * 4);
  w.lxm = (int32_t*)take(BH * 16 * 4);
  w.lsync = (uint32_t*)take(BH * 32 * 4);
  w.lstatus = (uint32_t*)take(64 * 4);
  if (ws) *ws = w;
  return off;
}

size_t noalloc_layout(const Dims& d, Workspace* ws, void* base) {
  const int64_t BH = d.BH, n = d.n, N = d.N;
  const int64_t Npad = (N + 31) & ~31;
  size_t off = 0;
  char* b = (char*)base;
  auto take = [&](size_t bytes) -> void* {
    void* p = b ? (void*)(b + off) : nullptr;
    off += align256(bytes);
    return p;
  };
  Workspace w{};
  w.C = (float*)take(BH * N * 64 * 4);
  w.R = take(BH * N * 64 * 2);
  w.nrm64 = (double*)take(BH * N * 8);
  w.nsplit = (uint16_t*)take(BH * N * 16);
  w.belong = (int32_t*)take(BH * n * 4);
  w.count = (int32_t*)take(BH * N * 4);
  w.Vt = (uint16_t*)take(BH * 64 * (int64_t)vt_stride((int)N) * 2);
  w.ginit = (float*)take(BH * Npad * 4);
  w.lxs = (double*)take(lloyd_exchange_rows(d) * 64 * 8);
  w.lxc = (int32_t*)take(lloyd_exchange_rows(d) * 4);
  w.lxm = (int32_t*)take(BH * 16 * 4);
  w.lsync = (uint32_t*)take(BH * 32 * 4);
  w.lstatus = (uint32_t*)take(64 * 4);
  if (ws) *ws = w;
  return off;
}

hipError_t launch_init(const Dims& d, const void* K, const float* init, float* C, void* R,
                       double* nrm64, uint16_t* nsplit, int32_t* mcount, hipStream_t st) {
  TimedLaunch timed("init", st);
  const dim3 grid(cdiv(d.N, 64), (unsigned)d.BH), block(256);
  if (d.dtype == 1)
    hipLaunchKernelGGL(k_init<BF16>, grid, block, 0, st, (const uint16_t*)K, init, d.n, d.N, C,
                       (uint16_t*)R, nrm64, nsplit, mcount);
  else
    hipLaunchKernelGGL(k_init<F32>, grid, block, 0, st, (const float*)K, init, d.n, d.N, C, (float*)R,
                       nrm64, nsplit, mcount);
  return hipGetLastError();
}

using AssignFn = void (*)(const uint16_t*, const uint16_t*, const uint16_t*, const double*, float*, int32_t*,
                          int32_t*, unsigned long long*, int, int, int, float, float, FusedUpdate);
struct AssignPlan {
  AssignFn kern;
  int64_t tpw, parts;
  bool fused;
};

// bf16 kernel choice and grid: one round of resident workgroups, the same
// number per slice, at most 16 tiles per wave (the LDS lists grow with tpw;
// the occupancy is taken at 16).
static AssignPlan plan_assign(const Dims& d, bool first) {
  const int64_t tiles = (d.n + 31) / 32;
  const int Npad = (d.N + 31) & ~31;
  // Npad <= 128: the register-resident kernel, one instantiation per block
  // count; the first round also with the partition sums
  static const AssignFn reg[3][4] = {
      {k_assign_reg<false, 1, false>, k_assign_reg<false, 2, false>, k_assign_reg<false, 3, false>,
       k_assign_reg<false, 4, false>},
      {k_assign_reg<true, 1, false>, k_assign_reg<true, 2, false>, k_assign_reg<true, 3, false>,
       k_assign_reg<true, 4, false>},
      {k_assign_reg<true, 1, true>, k_assign_reg<true, 2, true>, k_assign_reg<true, 3, true>,
       k_assign_reg<true, 4, true>}};
  const bool small = Npad <= kFusedG;
  AssignPlan p;
  p.kern = small ? reg[first][(Npad >> 5) - 1] : (first ? k_assign_bf16<true> : k_assign_bf16<false>);
  int64_t tpw = 16;
  while (tpw > 1 && assign_lds(d.N, (int)tpw) > kAssignLdsMax) --tpw;
  p.tpw = tiles_per_wave(tiles, d.BH, resident_wgs((const void*)p.kern, assign_lds(d.N, (int)tpw)), tpw);
  p.parts = cdiv(tiles, 4 * p.tpw);
  p.fused = first && small && p.parts <= kFusedP;
  if (p.fused) p.kern = reg[2][(Npad >> 5) - 1];
  return p;
}

int fused_first_parts(const Dims& d) {
  if (d.dtype != 1) return 0;
  const AssignPlan p = plan_assign(d, true);
  return p.fused ? (int)p.parts : 0;
}

hipError_t launch_assign(const Dims& d, const void* K, const void* R, const uint16_t* nsplit,
                         const double* nrm64, float* knorm, int32_t* belong, int32_t* mcount,
                         unsigned long long* mrec, bool first, const FusedUpdate& fu, int* parts_out,
                         hipStream_t st) {
  TimedLaunch timed(first ? "assign_first" : "assign", st);
  set_lds_limits();
  *parts_out = 0;
  if (d.dtype == 1) {
    // |MFMA fp32 accumulation error| <= (d + 4) 2^-24 * 2 * sum|terms| (each of the
    // d products and the three |r|^2 terms added with at most one rounding,
    // sequential model, 2x margin; the split itself is within 2^-24 |r|^2);
    // packing the register index into the low 4 mantissa bits moves a value by
    // < 2^(4 - 23) of its magnitude.
    const float cm = (float)(kD + 4) * 0x1p-23f * (1.0f + 0x1p-10f) * cert_widen();
    const float cp = 0x1p-19f * (1.0f + 0x1p-10f) * cert_widen();
    const AssignPlan p = plan_assign(d, first);
    if (p.fused) *parts_out = (int)p.parts;
    const dim3 grid((unsigned)p.parts, (unsigned)d.BH), block(256);
    const size_t lds = assign_lds(d.N, (int)p.tpw, p.fused);
    hipLaunchKernelGGL(p.kern, grid, block, lds, st, (const uint16_t*)K, (const uint16_t*)R, nsplit, nrm64, knorm,
                       belong, mcount, mrec, d.n, d.N, (int)p.tpw, cm, cp, fu);
  } else {
    const int kpw = 4;
    const dim3 grid(cdiv(d.n, 4 * kpw), (unsigned)d.BH), block(256);
    hipLaunchKernelGGL(k_assign_exact<F32>, grid, block, 0, st, (const float*)K, (const float*)R, nrm64,
                       belong, d.n, d.N, kpw);
  }
  return hipGetLastError();
}

hipError_t launch_part_finish(const Dims& d, int parts, const FusedUpdate& fu, double* S64,
                              int32_t* count, float* C, void* R, double* nrm64, uint16_t* nsplit,
                              hipStream_t st) {
  TimedLaunch timed("part_finish", st);
  if (parts < 1 || parts > kFusedP || d.N > kFusedG) return hipErrorInvalidValue;
  using FinishFn = void (*)(const double*, const int32_t*, const uint32_t*, int, double*, int32_t*, float*,
                            uint16_t*, double*, uint16_t*);
  static const FinishFn fns[kFusedP] = {k_part_finish<1>, k_part_finish<2>, k_part_finish<3>, k_part_finish<4>,
                                        k_part_finish<5>, k_part_finish<6>, k_part_finish<7>, k_part_finish<8>};
  const dim3 grid(cdiv(d.N, 32), (unsigned)d.BH), block(256);
  hipLaunchKernelGGL(fns[parts - 1], grid, block, 0, st, fu.Sp, fu.cntp, fu.pbits, d.N, S64, count, C,
                     (uint16_t*)R, nrm64, nsplit);
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

hipError_t launch_gsum(const Dims& d, int mode, const void* X, const int32_t* belong,
                       const unsigned long long* mrec, const int32_t* mcount_cur, int32_t* mcount_next,
                       double* S64, int32_t* count, float* out, void* R, double* nrm64, uint16_t* nsplit,
                       hipStream_t st) {
  TimedLaunch timed(mode == 0 ? "sums_full" : mode == 1 ? "sums_delta" : "valuesum", st);
  const dim3 grid(cdiv(d.N, kGsumG), (unsigned)d.BH), block(256);
  const size_t lds = 0;
  const uint16_t* Xb = (const uint16_t*)X;
  uint16_t* Rb = (uint16_t*)R;
  if (mode == 0)
    hipLaunchKernelGGL(k_gsum<0>, grid, block, lds, st, Xb, belong, d.n, d.N, S64, count, out, Rb, nrm64, nsplit,
                       0.f, 0);
  else if (mode == 1)
    hipLaunchKernelGGL(k_gdelta, grid, block, 0, st, Xb, mrec, mcount_cur, mcount_next, d.n, d.N, S64, count, out,
                       Rb, nrm64, nsplit);
  else
    hipLaunchKernelGGL(k_gsum<2>, grid, block, lds, st, Xb, belong, d.n, d.N, S64, count, out, Rb, nrm64, nsplit,
                       0.f, 0);
  return hipGetLastError();
}

static float clamp_sl2e(float scale) {
  const float s = fabsf(scale) * 1.4426950408889634f;
  return s < 1e-30f ? 1e-30f : s;
}

hipError_t launch_valuesum_prep(const Dims& d, const void* V, const int32_t* belong, const int32_t* count,
                                float scale, uint16_t* Vt, float* ginit, hipStream_t st) {
  TimedLaunch timed("valuesum", st);
  if (d.dtype != 1) return hipErrorInvalidValue;
  const dim3 grid(cdiv(d.N, kGsumG), (unsigned)d.BH), block(256);
  hipLaunchKernelGGL(k_gsum<3>, grid, block, 0, st, (const uint16_t*)V, belong, d.n, d.N, (double*)nullptr,
                     (int32_t*)count, ginit, Vt, (double*)nullptr, (uint16_t*)nullptr, 1.0f / clamp_sl2e(scale),
                     vt_stride(d.N));
  return hipGetLastError();
}

hipError_t launch_update(const Dims& d, const void* K, const int32_t* perm, const int32_t* goff,
                         const int32_t* count, float* C, void* R, double* nrm64, uint16_t* nsplit,
                         hipStream_t st) {
  TimedLaunch timed("update", st);
  const dim3 grid(cdiv(d.N, 4), (unsigned)d.BH), block(256);
  if (d.dtype == 1)
    hipLaunchKernelGGL((k_segsum<BF16, true>), grid, block, 0, st, (const uint16_t*)K, perm, goff, count,
                       d.n, d.N, C, (uint16_t*)R, nrm64, nsplit);
  else
    hipLaunchKernelGGL((k_segsum<F32, true>), grid, block, 0, st, (const float*)K, perm, goff, count, d.n,
                       d.N, C, (float*)R, nrm64, nsplit);
  return hipGetLastError();
}

hipError_t launch_valuesum(const Dims& d, const void* V, const int32_t* perm, const int32_t* goff,
                           const int32_t* count, float* vsum, hipStream_t st) {
  TimedLaunch timed("valuesum", st);
  const dim3 grid(cdiv(d.N, 4), (unsigned)d.BH), block(256);
  if (d.dtype == 1)
    hipLaunchKernelGGL((k_segsum<BF16, false>), grid, block, 0, st, (const uint16_t*)V, perm, goff, count,
                       d.n, d.N, vsum, (uint16_t*)nullptr, (double*)nullptr, (uint16_t*)nullptr);
  else
    hipLaunchKernelGGL((k_segsum<F32, false>), grid, block, 0, st, (const float*)V, perm, goff, count, d.n,
                       d.N, vsum, (float*)nullptr, (double*)nullptr, (uint16_t*)nullptr);
  return hipGetLastError();
}


hipError_t launch_attend_prep(const Dims& d, const float* centroid, const int32_t* count,
                              const float* vsum, float scale, uint16_t* Rq, uint16_t* Vt, float* ginit,
                              bool make_rq, hipStream_t st) {
  TimedLaunch timed("attend_prep", st);
  const int Npad = (d.N + 31) & ~31;
  const dim3 grid(cdiv(Npad, 64), (unsigned)d.BH), block(256);
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
    const uint32_t rsign = scale < 0.f ? 0x80008000u : 0u;
    using AttendFn = void (*)(const uint16_t*, const uint16_t*, const uint16_t*, const float*, int, int, int, float,
                              uint32_t, int, uint16_t*);
    static const AttendFn fns[8] = {k_attend_bf16<1>, k_attend_bf16<2>, k_attend_bf16<3>, k_attend_bf16<4>,
                                    k_attend_bf16<5>, k_attend_bf16<6>, k_attend_bf16<7>, k_attend_bf16<8>};
    const AttendFn fn = fns[((d.N + 31) >> 5) - 1];
    // one round of resident workgroups, the same number per slice
    const int64_t tpw = tiles_per_wave(tiles, d.BH, resident_wgs((const void*)fn, attend_lds(d.N)), 64);
    const dim3 grid(cdiv(tiles, 4 * tpw), (unsigned)d.BH), block(256);
    hipLaunchKernelGGL(fn, grid, block, attend_lds(d.N), st, (const uint16_t*)Q, (const uint16_t*)R, Vt, ginit, d.n,
                       d.N, vt_stride(d.N), clamp_sl2e(scale), rsign, (int)tpw, (uint16_t*)O);
  } else {
    const dim3 grid(cdiv(d.n, 256), (unsigned)d.BH), block(256);
    hipLaunchKernelGGL(k_attend_f32, grid, block, 0, st, (const float*)Q, centroid, count, vsum, d.n, d.N,
                       scale, (float*)O);
  }
  return hipGetLastError();
}

}  // namespace ga
