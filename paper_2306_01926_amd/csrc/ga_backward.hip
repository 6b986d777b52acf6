// gfx950 (MI355X) backward pass of group attention (bf16 storage, fp32
// accumulation).
//
// Forward (Eq. 3, Algorithm 1) for query i and group j with c_j members,
// representative r_j and value mean mu_j = vsum_j / c_j:
//   p_ij = scale q_i . r_j,   w_ij = c_j e^{p_ij} / sum_l c_l e^{p_il},
//   o_i = sum_j w_ij mu_j.
// The grouping (BELONG, COUNT) is piecewise constant in the keys, so the
// gradient treats it as fixed; r_j is the centroid (the mean of the member
// keys; bf16 rounding passed straight through) and mu_j the mean of the member
// values.  Given G = dL/dO:
//   dw_ij = G_i . mu_j,   D_i = sum_j w_ij dw_ij (= G_i . o_i),
//   dp_ij = w_ij (dw_ij - D_i),
//   dQ_i = scale sum_j dp_ij r_j,
//   dr_j = scale sum_i dp_ij q_i  ->  dK_k = dr_{a_k} / c_{a_k},
//   dmu_j = sum_i w_ij G_i        ->  dV_k = dmu_{a_k} / c_{a_k}.
//
// Kernels (N <= 256, padded to Npad = 32 NB groups).  N <= 128:
//   k_bwd_fused   per (slice, query chunk), 8 waves: the slice's group rows
//                 staged from the fp32 centroids and sums; per step of 128
//                 queries, each wave takes 16 (lane = query): MFMA scores,
//                 the group softmax, MFMA dw, D, dp, MFMA dQ, and writes its
//                 w and dp rows to LDS; then each wave adds the step into its
//                 part of dr += dp Q or dmu += w G (32 groups x 64 features,
//                 operands read back transposed), held in registers over the
//                 chunk
// N > 128 (two kernels; the group side recomputes the scores):
//   k_bwd_prep    per slice: R = bf16(centroid) rows and transposed, bf16
//                 value means, log2(count) (-inf for an empty group)
//   k_bwd_query   per 32-query tile (lane = query): the query side as above
//                 in three passes over the 32-group blocks (shift; sum and
//                 D; dp and dQ), recomputing the block's MFMAs; stores each
//                 query's softmax shift plus log2 of its sum (so that a
//                 weight is one exp2) and D
//   k_bwd_group   per (32-group block, query chunk): the same scores and dw
//                 in the transposed layout (lane = group), so that the dp and
//                 w registers are directly the A operand of the MFMA
//                 reductions; the four waves' partials are added in a fixed
//                 order ((w0 + w2) + (w1 + w3))
// Both:
//   k_bwd_finish  per group: the chunk partials added in a fixed order,
//                 scaled: scale dr / c and dmu / c, as bf16 rows (skipped
//                 with one chunk per slice: the chunk's kernel forms them)
//   k_bwd_keys    per key: the rows of its group to dK, dV (bf16)
// Every reduction has a fixed order, so repeated calls give identical bits.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include "ga_internal.h"

namespace ga {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kBs = 72;       // LDS row stride (bf16) of group rows and wave tiles
// Query chunks per slice in k_bwd_group: as few as give about kBwdTargetWgs
// workgroups (two per CU of a 256-CU MI355X at the kernel's 2 waves per SIMD),
// at most kBwdMaxChunks.  Each chunk writes its own partial sums, so fewer
// chunks mean fewer partial bytes and longer runs per workgroup setup.  A
// function of the shape only (the workspace size depends on it).
constexpr int kBwdMaxChunks = 8;
constexpr int64_t kBwdTargetWgs = 512;
int bwd_chunks(int64_t BH, int NB) {
  const int64_t c = (kBwdTargetWgs + NB * BH - 1) / (NB * BH);
  return (int)(c < 1 ? 1 : (c > kBwdMaxChunks ? kBwdMaxChunks : c));
}

__device__ __forceinline__ uint32_t bf16_bits(float x) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)x);  // round to nearest even
}
// two values rounded to bf16 (nearest even) in one v_cvt_pk_bf16_f32
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}
__device__ __forceinline__ f32x16 mfma(const u32x4& a, const u32x4& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0,
                                                 0, 0);
}
// LDS transpose read (ds_read_b64_tr_b16): within each 16-lane block, lane
// i receives element i % 4 of the 8-byte rows addressed by block lanes
// 4 j + i / 4, j = 0..3 (element j of the result from row j).  With block
// lane 4 j + s addressing row j at columns c0 + 4 s .. + 3, lane i gets
// column c0 + i of the four rows.
__device__ __forceinline__ u32x2 lds_tr16(const uint16_t* p) {
  const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)p);
  return __builtin_bit_cast(u32x2, v);
}
__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int v = 0; v < 16; ++v) z[v] = 0.f;
  return z;
}
// MFMA 32x32x16 layouts used below: the A operand of lane l is row l % 32, the
// B operand column l % 32, each with 8 contraction indices chosen by lane half
// h = l / 32; accumulator register v of lane l is row 8 (v / 4) + 4 h + v % 4,
// column l % 32.  Features are contracted in the order 32 h + 8 s .. + 7 at
// step s (both operands); groups or queries taken from accumulator registers
// are contracted in the order {16 u + 4 h + j, 16 u + 8 + 4 h + j : j < 4} at
// step u, the indices those registers hold.

// Padded slice layout of the workspace (all per slice bh):
//   R   [Npad][64] bf16,  RT [64][rts] bf16 (rts = Npad + 4),
//   MU  [Npad][64] bf16,  LC [Npad] f32.
// grid (Npad / 32, BH), 256 threads: one 32-group block; its R^T columns go
// through an LDS tile so that each transposed row segment is stored whole.
__global__ __launch_bounds__(256) void k_bwd_prep(const float* __restrict__ centroid, const int32_t* __restrict__ count,
                                                  const float* __restrict__ vsum, int N, int Npad, int rts,
                                                  uint16_t* __restrict__ R, uint16_t* __restrict__ RT,
                                                  uint16_t* __restrict__ MU, float* __restrict__ LC) {
  __shared__ uint16_t tt[64][32 + 2];
  const int64_t bh = blockIdx.y;
  const int g0 = 32 * blockIdx.x;
  // element x = threadIdx.x + 256 i: group g0 + x / 64, feature x % 64; every
  // load (rows clamped into the slice) is issued before any result is formed
  int cnt[8];
  float cv[8], sv[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int x = threadIdx.x + 256 * i, g = g0 + (x >> 6), c = x & 63;
    const int64_t row = bh * N + min(g, N - 1);
    cnt[i] = count[row];
    cv[i] = centroid[row * 64 + c];
    sv[i] = vsum[row * 64 + c];
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int x = threadIdx.x + 256 * i, g = g0 + (x >> 6), c = x & 63;
    const bool in = g < N;
    const int k = in ? cnt[i] : 0;
    const float mv = k > 0 ? sv[i] / (float)k : 0.f;
    const uint16_t rb = (uint16_t)bf16_bits(in ? cv[i] : 0.f);
    R[(bh * Npad + g) * 64 + c] = rb;
    tt[c][x >> 6] = rb;
    MU[(bh * Npad + g) * 64 + c] = (uint16_t)bf16_bits(mv);
    if (c == 0) LC[bh * Npad + g] = k > 0 ? log2f((float)k) : -INFINITY;
  }
  __syncthreads();
  for (int x = threadIdx.x; x < 64 * 16; x += 256) {
    const int c = x >> 4, p = x & 15;  // 16 pairs of groups per feature row
    *(uint32_t*)(RT + (bh * 64 + c) * rts + g0 + 2 * p) = (uint32_t)tt[c][2 * p] | ((uint32_t)tt[c][2 * p + 1] << 16);
  }
}

// Stage a slice's R rows (A or B operand rows), value-mean rows and the count
// logarithms in LDS.
template <int NB>
__device__ __forceinline__ void stage_groups(const uint16_t* __restrict__ R, const uint16_t* __restrict__ MU,
                                             const float* __restrict__ LC, int64_t bh, uint16_t* Rs, uint16_t* Ms,
                                             float* lc) {
  constexpr int Npad = NB * 32;
  for (int x = threadIdx.x; x < Npad * 8; x += 256) {
    const int row = x >> 3, ch = x & 7;
    *(u32x4*)(Rs + row * kBs + 8 * ch) = *(const u32x4*)(R + (bh * Npad + row) * 64 + 8 * ch);
    *(u32x4*)(Ms + row * kBs + 8 * ch) = *(const u32x4*)(MU + (bh * Npad + row) * 64 + 8 * ch);
  }
  for (int g = threadIdx.x; g < Npad; g += 256) lc[g] = LC[bh * Npad + g];
}

// lane (row, h) loads features 32 h .. 32 h + 31 of row `row` (clamped): the
// operand fragments of the 4 feature steps
__device__ __forceinline__ void load_row_frags(const uint16_t* __restrict__ X, int64_t row, u32x4 (&f)[4]) {
  const int h = (threadIdx.x & 63) >> 5;
#pragma unroll
  for (int s = 0; s < 4; ++s) f[s] = *(const u32x4*)(X + row * 64 + 32 * h + 8 * s);
}

// grid (ceil(tiles / (4 tpw)), BH), 256 threads: wave tiles of 32 queries.
template <int NB>
__global__ __launch_bounds__(256) void k_bwd_query(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ G,
                                                   const uint16_t* __restrict__ R, const uint16_t* __restrict__ RT,
                                                   const uint16_t* __restrict__ MU, const float* __restrict__ LC,
                                                   int n, int rts, float scale, float sl2e, int tpw,
                                                   uint16_t* __restrict__ dQ, float2* __restrict__ stats) {
  constexpr int Npad = NB * 32;
  __shared__ __attribute__((aligned(16))) uint16_t Rs[Npad * kBs];
  __shared__ __attribute__((aligned(16))) uint16_t Ms[Npad * kBs];
  __shared__ __attribute__((aligned(16))) uint16_t RTs[64 * (Npad + 4)];
  __shared__ float lc[Npad];
  __shared__ __attribute__((aligned(16))) uint16_t Ot[4][32 * kBs];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5, q = lane & 31;
  const int64_t bh = blockIdx.y;
  stage_groups<NB>(R, MU, LC, bh, Rs, Ms, lc);
  for (int x = tid; x < 64 * (Npad / 4); x += 256) {
    const int row = x / (Npad / 4), ch = x % (Npad / 4);
    *(u32x2*)(RTs + row * (Npad + 4) + 4 * ch) = *(const u32x2*)(RT + (bh * 64 + row) * rts + 4 * ch);
  }
  __syncthreads();
  const int64_t ntiles = ((int64_t)n + 31) / 32;
  const int64_t t0 = ((int64_t)blockIdx.x * 4 + wave) * tpw;
  const uint16_t* Qb = Q + bh * (int64_t)n * 64;
  const uint16_t* Gb = G + bh * (int64_t)n * 64;
  uint16_t* Ow = Ot[wave];
  const int64_t tend = min(t0 + tpw, ntiles);
  // the next tile's rows load while the current tile is processed
  // (unconditional, rows clamped, so the loads stay ahead of the tile's work)
  u32x4 qn[4], gn[4];
  load_row_frags(Qb, min(t0 * 32 + q, (int64_t)n - 1), qn);
  load_row_frags(Gb, min(t0 * 32 + q, (int64_t)n - 1), gn);
  for (int64_t t = t0; t < tend; ++t) {
    const int64_t qi = t * 32 + q;
    u32x4 qf[4], gf[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      qf[s] = qn[s];
      gf[s] = gn[s];
    }
    load_row_frags(Qb, min(qi + 32, (int64_t)n - 1), qn);
    load_row_frags(Gb, min(qi + 32, (int64_t)n - 1), gn);
    __builtin_amdgcn_sched_barrier(0);
    // block b's scores r_g . q and dw_gq = mu_g . G_q (rows g, column q)
    auto block_mfma = [&](int b, f32x16& a, f32x16& d) __attribute__((always_inline)) {
      a = zero16();
      d = zero16();
      const uint16_t* rr = Rs + (32 * b + q) * kBs + 32 * h;
      const uint16_t* mr = Ms + (32 * b + q) * kBs + 32 * h;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        a = mfma(*(const u32x4*)(rr + 8 * s), qf[s], a);
        d = mfma(*(const u32x4*)(mr + 8 * s), gf[s], d);
      }
    };
    // dQ^T[f][q] += sum_g r_gf dp_gq over block b: A = R^T rows (features), B = dp from the registers
    f32x16 o0 = zero16(), o1 = zero16();
    auto dq_block = [&](int b, const float (&dp)[16]) __attribute__((always_inline)) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const u32x4 bf = {pack2(dp[8 * u], dp[8 * u + 1]), pack2(dp[8 * u + 2], dp[8 * u + 3]),
                          pack2(dp[8 * u + 4], dp[8 * u + 5]), pack2(dp[8 * u + 6], dp[8 * u + 7])};
        const int gcol = 32 * b + 16 * u + 4 * h;
        const uint16_t* r0 = RTs + q * (Npad + 4) + gcol;
        const uint16_t* r1 = RTs + (32 + q) * (Npad + 4) + gcol;
        const u32x2 a0l = *(const u32x2*)r0, a0h = *(const u32x2*)(r0 + 8);
        const u32x2 a1l = *(const u32x2*)r1, a1h = *(const u32x2*)(r1 + 8);
        o0 = mfma(u32x4{a0l[0], a0l[1], a0h[0], a0h[1]}, bf, o0);
        o1 = mfma(u32x4{a1l[0], a1l[1], a1h[0], a1h[1]}, bf, o1);
      }
    };
    float Ms_, inv, Dq, Lq;  // Lq: the shift plus log2 of the sum (+inf if every group is empty)
    {
      // more groups than fit in registers: three passes over the blocks
      // (shift; sum and D; dp and dQ), the MFMAs recomputed in each
      float M = -INFINITY;
      for (int b = 0; b < NB; ++b) {
        f32x16 a, d;
        block_mfma(b, a, d);
#pragma unroll
        for (int v = 0; v < 16; ++v) M = fmaxf(M, fmaf(a[v], sl2e, lc[32 * b + 8 * (v >> 2) + 4 * h + (v & 3)]));
      }
      M = fmaxf(M, __shfl_xor(M, 32));
      const bool any = M != -INFINITY;
      Ms_ = any ? M : 0.f;
      float S = 0.f, SD = 0.f;
      for (int b = 0; b < NB; ++b) {
        f32x16 a, d;
        block_mfma(b, a, d);
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float e =
              __builtin_amdgcn_exp2f(fmaf(a[v], sl2e, lc[32 * b + 8 * (v >> 2) + 4 * h + (v & 3)]) - Ms_);
          S += e;
          SD = fmaf(e, d[v], SD);
        }
      }
      S += __shfl_xor(S, 32);
      SD += __shfl_xor(SD, 32);
      inv = any ? 1.0f / S : 0.f;
      Lq = any ? Ms_ + log2f(S) : INFINITY;
      Dq = SD * inv;
      for (int b = 0; b < NB; ++b) {
        f32x16 a, d;
        block_mfma(b, a, d);
        float dp[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float w =
              __builtin_amdgcn_exp2f(fmaf(a[v], sl2e, lc[32 * b + 8 * (v >> 2) + 4 * h + (v & 3)]) - Ms_) * inv;
          dp[v] = w * (d[v] - Dq);
        }
        dq_block(b, dp);
      }
    }
    // dQ rows through the wave's LDS tile: lane (q, h) holds features 8 k + 4 h + j
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      *(u32x2*)(Ow + q * kBs + 8 * k + 4 * h) = u32x2{pack2(scale * o0[4 * k], scale * o0[4 * k + 1]),
                                                      pack2(scale * o0[4 * k + 2], scale * o0[4 * k + 3])};
      *(u32x2*)(Ow + q * kBs + 32 + 8 * k + 4 * h) = u32x2{pack2(scale * o1[4 * k], scale * o1[4 * k + 1]),
                                                           pack2(scale * o1[4 * k + 2], scale * o1[4 * k + 3])};
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int row = 8 * k + (lane >> 3), ch = lane & 7;
      const int64_t qo = t * 32 + row;
      if (qo < n) *(u32x4*)(dQ + (bh * (int64_t)n + qo) * 64 + 8 * ch) = *(const u32x4*)(Ow + row * kBs + 8 * ch);
    }
    if (h == 0 && qi < n) stats[bh * (int64_t)n + qi] = make_float2(Lq, Dq);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

// 1-D grid of ceil(NB chunks BH / 8) * 8 workgroups, 256 threads: work
// item (bh, chunk, b) is group block b of slice bh over query chunk c (tiles
// [c T / chunks, (c + 1) T / chunks), wave w takes every 4th).  Items are
// handed to the XCDs in contiguous ranges (workgroup x runs on XCD x % 8), so
// the NB group blocks that read the same query and dO rows run together on
// one XCD and share its L2.
// part[bh][c][0/1][g][f] = this chunk's sum_i dp_gi q_if / sum_i w_gi G_if.
template <int NB>
__global__ __launch_bounds__(256) void k_bwd_group(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ G,
                                                   const uint16_t* __restrict__ R, const uint16_t* __restrict__ MU,
                                                   const float* __restrict__ LC, const float2* __restrict__ stats,
                                                   int n, int64_t BH, int chunks, float sl2e,
                                                   float* __restrict__ part, const int32_t* __restrict__ count,
                                                   int N, float scale, uint16_t* __restrict__ gk,
                                                   uint16_t* __restrict__ gv) {
  constexpr int Npad = NB * 32;
  // the waves' query tiles; after the loop the same bytes hold two partial
  // slots [2][2][32][64] (waves 0, 1 write, waves 2, 3 add: fixed order)
  constexpr int kTiles = 8 * 32 * kBs * 2, kRed = 2 * 2 * 32 * 64 * 4;
  __shared__ __attribute__((aligned(16))) unsigned char lds[kTiles > kRed ? kTiles : kRed];
  uint16_t* Qt = (uint16_t*)lds;  // [4][32][kBs]
  uint16_t* Gt = Qt + 4 * 32 * kBs;
  float* red = (float*)lds;
  __shared__ __attribute__((aligned(16))) float2 st[4][32];  // (Lq, D) of the wave's tile queries
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5, gl = lane & 31;
  const int64_t item = (int64_t)(blockIdx.x % 8) * (gridDim.x / 8) + blockIdx.x / 8;
  if (item >= NB * chunks * BH) return;  // grid padding (whole workgroup)
  const int b = (int)(item % NB), chunk = (int)(item / NB % chunks);
  const int64_t bh = item / (NB * chunks);
  const int64_t ntiles = ((int64_t)n + 31) / 32;
  const int64_t c0 = chunk * ntiles / chunks, c1 = (chunk + 1) * ntiles / chunks;
  const uint16_t* Qb = Q + bh * (int64_t)n * 64;
  const uint16_t* Gb = G + bh * (int64_t)n * 64;
  const int g = 32 * b + gl;  // this lane's group (MFMA column / A-operand row)
  const float lcg = LC[bh * Npad + g];
  // the lane's group row (features 32 h ..) of R and of the value means: the
  // B operands of every tile's score and dw MFMAs
  u32x4 rf[4], mf[4];
  load_row_frags(R + bh * (int64_t)Npad * 64, g, rf);
  load_row_frags(MU + bh * (int64_t)Npad * 64, g, mf);
  uint16_t *Qw = Qt + wave * 32 * kBs, *Gw = Gt + wave * 32 * kBs;
  f32x16 dr0 = zero16(), dr1 = zero16(), dm0 = zero16(), dm1 = zero16();
  // the wave's next tile (its query stats, then its rows) loads while the
  // current one is processed
  const float2* statb = stats + bh * (int64_t)n;
  float2 sn = statb[min((c0 + wave) * 32 + gl, (int64_t)n - 1)];
  u32x4 qn[4], gn[4];
  load_row_frags(Qb, min((c0 + wave) * 32 + gl, (int64_t)n - 1), qn);
  load_row_frags(Gb, min((c0 + wave) * 32 + gl, (int64_t)n - 1), gn);
  for (int64_t t = c0 + wave; t < c1; t += 4) {
    // lane (row = query gl, h): its query's features as A fragments, also
    // kept row-major in the wave's tile for the transposed reads below
    const int64_t qi = t * 32 + gl;
    u32x4 qf[4], gf[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      qf[s] = qn[s];
      gf[s] = gn[s];
    }
    const float2 sc = sn;
    // unconditional (rows clamped; past the chunk it loads a row again), so
    // the loads stay in this block, ahead of the tile's work
    sn = statb[min(qi + 128, (int64_t)n - 1)];
    load_row_frags(Qb, min(qi + 128, (int64_t)n - 1), qn);
    load_row_frags(Gb, min(qi + 128, (int64_t)n - 1), gn);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      *(u32x4*)(Qw + gl * kBs + 32 * h + 8 * s) = qf[s];
      *(u32x4*)(Gw + gl * kBs + 32 * h + 8 * s) = gf[s];
    }
    if (h == 0) st[wave][gl] = qi < n ? sc : make_float2(INFINITY, 0.f);  // padded query: w = 0
    // scores and dw with queries as rows, groups as columns
    f32x16 x = zero16(), dw = zero16();
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      x = mfma(qf[s], rf[s], x);
      dw = mfma(gf[s], mf[s], dw);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // register v: query 8 (v / 4) + 4 h + v % 4 of the tile (two queries'
    // (Lq, D) per 16-byte read); w = 2^(p log2 e + log2 c - Lq)
    float w[16], dp[16];
#pragma unroll
    for (int a = 0; a < 4; ++a) {
#pragma unroll
      for (int p2 = 0; p2 < 2; ++p2) {
        const float4 sq = *(const float4*)&st[wave][8 * a + 4 * h + 2 * p2];
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          const int v = 4 * a + 2 * p2 + k;
          w[v] = __builtin_amdgcn_exp2f(fmaf(x[v], sl2e, lcg) - (k ? sq.z : sq.x));
          dp[v] = w[v] * (dw[v] - (k ? sq.w : sq.y));
        }
      }
    }
    // dr[g][f] += sum_q dp[g][q] Q[q][f]; dmu[g][f] += sum_q w[g][q] G[q][f]
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const u32x4 adp = {pack2(dp[8 * u], dp[8 * u + 1]), pack2(dp[8 * u + 2], dp[8 * u + 3]),
                         pack2(dp[8 * u + 4], dp[8 * u + 5]), pack2(dp[8 * u + 6], dp[8 * u + 7])};
      const u32x4 aw = {pack2(w[8 * u], w[8 * u + 1]), pack2(w[8 * u + 2], w[8 * u + 3]),
                        pack2(w[8 * u + 4], w[8 * u + 5]), pack2(w[8 * u + 6], w[8 * u + 7])};
      // B operands: lane (feature 32 fb + gl, h) takes queries r0 .. r0 + 3,
      // r0 + 8 .. r0 + 11 of the tile (the k order of the A operand), two
      // transpose reads each: block lane 4 j + s addresses query row r0 + j
      // (then r0 + 8 + j) at features 32 fb + 16 (lane / 16 % 2) + 4 s
      const int r0 = 16 * u + 4 * h;
      const int tro = (r0 + ((lane & 15) >> 2)) * kBs + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
      u32x4 bq[2], bg[2];
#pragma unroll
      for (int fb = 0; fb < 2; ++fb) {
        const u32x2 q0 = lds_tr16(Qw + tro + 32 * fb), q1 = lds_tr16(Qw + tro + 8 * kBs + 32 * fb);
        const u32x2 g0 = lds_tr16(Gw + tro + 32 * fb), g1 = lds_tr16(Gw + tro + 8 * kBs + 32 * fb);
        bq[fb] = u32x4{q0[0], q0[1], q1[0], q1[1]};
        bg[fb] = u32x4{g0[0], g0[1], g1[0], g1[1]};
      }
      dr0 = mfma(adp, bq[0], dr0);
      dr1 = mfma(adp, bq[1], dr1);
      dm0 = mfma(aw, bg[0], dm0);
      dm1 = mfma(aw, bg[1], dm1);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  // accumulator register v of lane (col = feature gl, h): group row 8 (v / 4) + 4 h + v % 4
  __syncthreads();  // every wave is done with the tiles
  float* rw = red + (wave & 1) * 2 * 32 * 64;
  for (int pass = 0; pass < 2; ++pass) {
    if ((wave >> 1) == pass) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int gr = 8 * (v >> 2) + 4 * h + (v & 3);
        float* r0 = rw + gr * 64 + gl;
        float* r1 = rw + 32 * 64 + gr * 64 + gl;
        if (pass == 0) {
          r0[0] = dr0[v];
          r0[32] = dr1[v];
          r1[0] = dm0[v];
          r1[32] = dm1[v];
        } else {
          r0[0] += dr0[v];
          r0[32] += dr1[v];
          r1[0] += dm0[v];
          r1[32] += dm1[v];
        }
      }
    }
    __syncthreads();
  }
  if (chunks == 1) {
    // the only chunk: the rows k_bwd_finish would form from it (the same
    // operations: its sum over one partial is 0 + s = s)
    for (int e = tid; e < 32 * 64; e += 256) {
      const int g = 32 * b + (e >> 6);
      if (g >= N) continue;
      const float sr = 0.f + (red[e] + red[2 * 32 * 64 + e]);
      const float sm = 0.f + (red[32 * 64 + e] + red[3 * 32 * 64 + e]);
      const int cnt = count[bh * N + g];
      gk[(bh * Npad + g) * 64 + (e & 63)] = (uint16_t)bf16_bits(cnt > 0 ? scale * sr / (float)cnt : 0.f);
      gv[(bh * Npad + g) * 64 + (e & 63)] = (uint16_t)bf16_bits(cnt > 0 ? sm / (float)cnt : 0.f);
    }
    return;
  }
  float* out = part + ((bh * chunks + chunk) * 2) * (int64_t)Npad * 64;
  for (int x = tid; x < 2 * 32 * 64; x += 256) {
    const int k = x / (32 * 64), e = x % (32 * 64);
    const float s = red[k * 32 * 64 + e] + red[2 * 32 * 64 + k * 32 * 64 + e];  // (w0 + w2) + (w1 + w3)
    out[(int64_t)k * Npad * 64 + 32 * b * 64 + e] = s;
  }
}

// ---------------------------------------------------------------- fused path
// N <= 128 (NB <= 4 blocks of 32 groups): one launch does the work of
// k_bwd_prep, k_bwd_query and k_bwd_group.  A workgroup of 8 waves (two per
// SIMD) takes a slice's query chunk in steps of 128 queries:
//   1. each wave takes 16 of them (lane = query): MFMA 16x16x32 scores and dw
//      against the slice's groups, the group softmax, D, dp, MFMA dQ; it
//      writes its w and dp rows (every group) and its q and dO rows to LDS;
//   2. after a barrier, wave (t, p) adds the step's 128 queries into its part
//      of the sums: t = 0 dr += dp Q, t = 1 dmu += w dO, for the 32 groups of
//      tile column block p and all 64 features (MFMA 32x32x16, both operands
//      read with transpose reads: lane = group, lane = feature);
// then a second barrier.  Each (sum, group, feature) has one owning wave, so
// the chunk's sums need no reduction across waves.
//
// Group order in the w / dp rows: lane (query, kq) holds groups
// 16 b + 4 kq + v (block b of 16, register v of a score accumulator), written
// contiguously at column 8 NB kq + 4 b + v; fcol_group() inverts that.
__device__ __forceinline__ int fcol_group(int c, int nb8) {
  const int kq = c / nb8, r = c % nb8;
  return 16 * (r >> 2) + 4 * kq + (r & 3);
}
typedef float f32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ f32x4 mfma16(const u32x4& a, const u32x4& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0,
                                                 0, 0);
}
constexpr int kFusedWgs = 256;  // workgroups to aim for: one per MI355X compute unit
constexpr int kStepQ = 128;     // queries per step (8 waves x 16)

// LDS rows without padding: each row's 16-byte chunks are permuted by XOR
// with a function of the row, chosen so that the accesses of the fused kernel
// touch each bank once per 256-byte cycle (16 lanes of a 16-byte access, 32
// lanes of an 8-byte or transpose access):
//   fR: 128-byte rows of R / value means, read 16 rows x one chunk (scores)
//       and 8 rows x two chunks (transpose reads for dQ);
//   fQ: 128-byte rows (q / dO, and w / dp rows of 64), written 16 rows x one
//       chunk, read 4 rows x 4 chunks (transpose reads);
//   fW: 256-byte w / dp rows, the same accesses.
__device__ __forceinline__ int fR(int r) { return (((r >> 1) & 3) << 1) | ((r >> 3) & 1); }
__device__ __forceinline__ int fQ(int r) { return (((r >> 1) & 1) << 2) | (((r >> 2) & 1) << 1) | ((r >> 3) & 1); }
__device__ __forceinline__ int fW(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }
// element offset of column c (bf16, a multiple of 4) of row r: rows of len elements, chunk permutation f
__device__ __forceinline__ int swz(int r, int len, int c, int f) { return r * len + ((((c >> 3) ^ f) << 3) | (c & 7)); }

// max / sum over the lanes l, l ^ 16, l ^ 32, l ^ 48 with the cross-row lane
// swaps of gfx950 (VALU; each swap leaves a lane its own value and its
// partner's, in row order, so all four lanes get the same bits)
__device__ __forceinline__ float xrow_max(float v) {
  auto t = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(t[0]), __uint_as_float(t[1]));
  t = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(t[0]), __uint_as_float(t[1]));
}
__device__ __forceinline__ float xrow_sum(float v) {
  auto t = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(t[0]) + __uint_as_float(t[1]);
  t = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(t[0]) + __uint_as_float(t[1]);
}

// Query chunks per slice of the fused kernel: about kFusedWgs workgroups, each
// with at least two steps.  A function of the shape only.
int fused_chunks(int64_t BH, int n) {
  const int64_t steps = ((int64_t)n + kStepQ - 1) / kStepQ;
  int64_t c = (kFusedWgs + BH - 1) / BH;
  const int64_t cmax = steps / 2 > 1 ? steps / 2 : 1;
  return (int)(c < cmax ? c : cmax);
}

// 1-D grid of BH chunks workgroups, 512 threads.  Workgroup (bh, c) takes the
// steps [c S / chunks, (c + 1) S / chunks) of slice bh; it writes its sums of
// dp q and w dO per group to part[bh][c] (or, the only chunk, the rows
// k_bwd_finish would form from them to gk / gv).
template <int NB>
__global__ __launch_bounds__(512) void k_bwd_fused(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ G,
                                                   const float* __restrict__ centroid,
                                                   const int32_t* __restrict__ count, const float* __restrict__ vsum,
                                                   int n, int N, int chunks, float scale, float sl2e,
                                                   uint16_t* __restrict__ dQ, float* __restrict__ part,
                                                   uint16_t* __restrict__ gk, uint16_t* __restrict__ gv) {
  constexpr int Npad = NB * 32, NB16 = 2 * NB, nb8 = 8 * NB;
  // LDS rows without padding, their chunks permuted by fR (R, value means),
  // fQ (q / dO rows) and fWP (w / dp rows: fW for 256-byte rows, fQ for 128)
  constexpr int kWs = Npad <= 64 ? 64 : 128;  // row length (bf16) of the w / dp rows
  auto fWP = [](int r) { return kWs == 128 ? fW(r) : fQ(r); };
  __shared__ __attribute__((aligned(16))) uint16_t Rs[Npad * 64];
  __shared__ __attribute__((aligned(16))) uint16_t Ms[Npad * 64];
  __shared__ __attribute__((aligned(16))) float lc[Npad];
  __shared__ __attribute__((aligned(16))) uint16_t WP[2][kStepQ * kWs];  // dp, w rows of the step
  __shared__ __attribute__((aligned(16))) uint16_t QT[2][kStepQ * 64];  // q, dO rows of the step
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i = lane & 15, kq = lane >> 4;  // MFMA 16x16x32 lane: row / column i, k-group kq
  const int64_t bh = blockIdx.x / chunks;
  const int chunk = blockIdx.x % chunks;

  // the slice's group rows, as k_bwd_prep forms them: R = bf16(centroid),
  // value means bf16(vsum / count) (0 for an empty group), log2(count)
  // (-inf for an empty group); thread x: group x / 16, features 4 (x % 16) ..
  {
    constexpr int kIt = (Npad * 16 + 511) / 512;
    float4 cv[kIt], sv[kIt];
    int cnt[kIt];
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
      const int x = min(tid + 512 * it, Npad * 16 - 1), g = x >> 4;
      const int64_t row = bh * N + min(g, N - 1);
      cnt[it] = count[row];
      cv[it] = *(const float4*)(centroid + row * 64 + 4 * (x & 15));
      sv[it] = *(const float4*)(vsum + row * 64 + 4 * (x & 15));
    }
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
      const int x = tid + 512 * it, g = x >> 4, c = 4 * (x & 15);
      if (x >= Npad * 16) break;
      const bool in = g < N;
      const int k = in ? cnt[it] : 0;
      const float4 r = in ? cv[it] : make_float4(0.f, 0.f, 0.f, 0.f);
      float4 m = make_float4(0.f, 0.f, 0.f, 0.f);
      if (k > 0)
        m = make_float4(sv[it].x / (float)k, sv[it].y / (float)k, sv[it].z / (float)k, sv[it].w / (float)k);
      *(u32x2*)(Rs + swz(g, 64, c, fR(g))) = u32x2{pack2(r.x, r.y), pack2(r.z, r.w)};
      *(u32x2*)(Ms + swz(g, 64, c, fR(g))) = u32x2{pack2(m.x, m.y), pack2(m.z, m.w)};
      if (c == 0) lc[g] = k > 0 ? log2f((float)k) : -INFINITY;
    }
  }
  __syncthreads();

  const int64_t nsteps = ((int64_t)n + kStepQ - 1) / kStepQ;
  const int64_t s0 = chunk * nsteps / chunks, s1 = (chunk + 1) * nsteps / chunks;
  const uint16_t* Qb = Q + bh * (int64_t)n * 64;
  const uint16_t* Gb = G + bh * (int64_t)n * 64;
  // the fold's part: t = 0 dr (dp, q), 1 dmu (w, dO); columns 32 p .. of the w / dp rows
  const int ft = wave >> 2, fp = wave & 3;
  const uint16_t* fA = WP[ft];
  const uint16_t* fB = QT[ft];
  f32x16 acc0 = zero16(), acc1 = zero16();  // features 0..31, 32..63
  // transpose-read addressing (16-lane block: lane 4 j + s reads row j at columns + 4 s)
  const int trr = (lane & 15) >> 2, trc = 16 * ((lane >> 4) & 1) + 4 * (lane & 3), h = lane >> 5;
  // lane (i, kq): features 8 kq .. and 32 + 8 kq .. of its query row
  auto load_q = [&](const uint16_t* X, int64_t row, u32x4 (&f)[2]) __attribute__((always_inline)) {
    f[0] = *(const u32x4*)(X + row * 64 + 8 * kq);
    f[1] = *(const u32x4*)(X + row * 64 + 32 + 8 * kq);
  };
  // per-lane LDS offsets (the rows' chunk permutations); the loops add
  // whole rows, which keep the permutation
  const int oS0 = swz(i, 64, 8 * kq, fR(i)), oS1 = swz(i, 64, 32 + 8 * kq, fR(i));  // score / dw A operands
  int oT[4];  // dQ A operands: rows 4 kq + trr (+ 32 u, + 16), features 16 fb + 4 (lane % 4)
#pragma unroll
  for (int fb = 0; fb < 4; ++fb) oT[fb] = swz(4 * kq + trr, 64, 16 * fb + 4 * (lane & 3), fR(4 * kq + trr));
  const int row = 16 * wave + i;  // this lane's row of the step
  const int oQ0 = swz(row, 64, 8 * kq, fQ(row)), oQ1 = swz(row, 64, 32 + 8 * kq, fQ(row));  // q / dO rows
  // the reductions' transpose reads: rows 8 h + trr (+ 4, + 16 ks)
  const int ra = 8 * h + trr;
  const int oA[2] = {swz(ra, kWs, 32 * fp + trc, fWP(ra)), swz(ra + 4, kWs, 32 * fp + trc, fWP(ra + 4))};
  const int oB[4] = {swz(ra, 64, trc, fQ(ra)), swz(ra + 4, 64, trc, fQ(ra + 4)), swz(ra, 64, 32 + trc, fQ(ra)),
                     swz(ra + 4, 64, 32 + trc, fQ(ra + 4))};
  u32x4 qn[2], gn[2];
  {
    const int64_t r = min(s0 * kStepQ + 16 * wave + i, (int64_t)n - 1);
    load_q(Qb, r, qn);
    load_q(Gb, r, gn);
  }
  for (int64_t st = s0; st < s1; ++st) {
    const int64_t qi = st * kStepQ + 16 * wave + i;  // this lane's query
    u32x4 qf[2] = {qn[0], qn[1]}, gf[2] = {gn[0], gn[1]};
    {
      const int64_t r = min(qi + kStepQ, (int64_t)n - 1);
      load_q(Qb, r, qn);
      load_q(Gb, r, gn);
    }
    __builtin_amdgcn_sched_barrier(0);
    // ---- 1. this wave's 16 queries against every group
    // scores (log2 domain, count bias added): x[b][v] is group 16 b + 4 kq + v
    f32x4 x[NB16], dw[NB16];
#pragma unroll
    for (int b = 0; b < NB16; ++b) {
      x[b] = f32x4{0.f, 0.f, 0.f, 0.f};
      dw[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int o = (s ? oS1 : oS0) + 16 * b * 64;
        x[b] = mfma16(*(const u32x4*)(Rs + o), qf[s], x[b]);
        dw[b] = mfma16(*(const u32x4*)(Ms + o), gf[s], dw[b]);
      }
      const float4 l4 = *(const float4*)(lc + 16 * b + 4 * kq);
      x[b][0] = fmaf(x[b][0], sl2e, l4.x);
      x[b][1] = fmaf(x[b][1], sl2e, l4.y);
      x[b][2] = fmaf(x[b][2], sl2e, l4.z);
      x[b][3] = fmaf(x[b][3], sl2e, l4.w);
    }
    float M = -INFINITY;
#pragma unroll
    for (int b = 0; b < NB16; ++b)
#pragma unroll
      for (int v = 0; v < 4; ++v) M = fmaxf(M, x[b][v]);
    M = xrow_max(M);
    const bool any = M != -INFINITY;  // some group is non-empty
    const float Ms_ = any ? M : 0.f;
    float S = 0.f, SD = 0.f;
#pragma unroll
    for (int b = 0; b < NB16; ++b)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        x[b][v] = __builtin_amdgcn_exp2f(x[b][v] - Ms_);  // 0 for an empty group
        S += x[b][v];
        SD = fmaf(x[b][v], dw[b][v], SD);
      }
    S = xrow_sum(S);
    SD = xrow_sum(SD);
    // a padded query (past n) gets weight 0: it adds nothing to the sums
    const float inv = any && qi < n ? 1.0f / S : 0.f;
    const float Dq = SD * inv;  // D = sum_g w dw
    uint32_t pw[2 * NB16], pd[2 * NB16];
#pragma unroll
    for (int b = 0; b < NB16; ++b) {
      float w[4], dp[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        w[v] = x[b][v] * inv;
        dp[v] = w[v] * (dw[b][v] - Dq);
      }
      pw[2 * b] = pack2(w[0], w[1]);
      pw[2 * b + 1] = pack2(w[2], w[3]);
      pd[2 * b] = pack2(dp[0], dp[1]);
      pd[2 * b + 1] = pack2(dp[2], dp[3]);
    }
    // dQ^T[f][q] = sum_g r_gf dp_gq over 32-group steps u (blocks 2 u, 2 u + 1):
    // A = R^T (transpose reads: groups 32 u + 4 kq + 0..3, then + 16), B = dp
    f32x4 o[4];
#pragma unroll
    for (int fb = 0; fb < 4; ++fb) o[fb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      const u32x4 bd = {pd[4 * u], pd[4 * u + 1], pd[4 * u + 2], pd[4 * u + 3]};
#pragma unroll
      for (int fb = 0; fb < 4; ++fb) {
        const u32x2 al = lds_tr16(Rs + oT[fb] + 32 * u * 64);
        const u32x2 ah = lds_tr16(Rs + oT[fb] + (32 * u + 16) * 64);
        o[fb] = mfma16(u32x4{al[0], al[1], ah[0], ah[1]}, bd, o[fb]);
      }
    }
    // dQ: lane (query i, kq) holds features 16 fb + 4 kq + v
    if (qi < n) {
#pragma unroll
      for (int fb = 0; fb < 4; ++fb)
        *(u32x2*)(dQ + (bh * (int64_t)n + qi) * 64 + 16 * fb + 4 * kq) =
            u32x2{pack2(scale * o[fb][0], scale * o[fb][1]), pack2(scale * o[fb][2], scale * o[fb][3])};
    }
    // the step's rows for the reductions
#pragma unroll
    for (int c = 0; c < NB; ++c) {
      const int o = swz(row, kWs, nb8 * kq + 8 * c, fWP(row));
      *(u32x4*)(WP[0] + o) = u32x4{pd[4 * c], pd[4 * c + 1], pd[4 * c + 2], pd[4 * c + 3]};
      *(u32x4*)(WP[1] + o) = u32x4{pw[4 * c], pw[4 * c + 1], pw[4 * c + 2], pw[4 * c + 3]};
    }
    *(u32x4*)(QT[0] + oQ0) = qf[0];
    *(u32x4*)(QT[0] + oQ1) = qf[1];
    *(u32x4*)(QT[1] + oQ0) = gf[0];
    *(u32x4*)(QT[1] + oQ1) = gf[1];
    __syncthreads();
    // ---- 2. wave (t, p): sums over the step's queries, 16 per MFMA step:
    // A = the w / dp rows read transposed (lane = column 32 p + m, queries
    // 16 ks + 8 h + 0..7), B = the q / dO rows read transposed (lane = feature)
    if (fp < NB) {
#pragma unroll
      for (int ks = 0; ks < kStepQ / 16; ++ks) {
        const u32x2 a0 = lds_tr16(fA + oA[0] + 16 * ks * kWs), a1 = lds_tr16(fA + oA[1] + 16 * ks * kWs);
        const u32x2 b0 = lds_tr16(fB + oB[0] + 16 * ks * 64), b1 = lds_tr16(fB + oB[1] + 16 * ks * 64);
        const u32x2 b2 = lds_tr16(fB + oB[2] + 16 * ks * 64), b3 = lds_tr16(fB + oB[3] + 16 * ks * 64);
        const u32x4 av = {a0[0], a0[1], a1[0], a1[1]};
        acc0 = mfma(av, u32x4{b0[0], b0[1], b1[0], b1[1]}, acc0);
        acc1 = mfma(av, u32x4{b2[0], b2[1], b3[0], b3[1]}, acc1);
      }
    }
    __syncthreads();
  }
  // wave (t, p): register v of lane (feature f, h) is column 32 p + 8 (v / 4) + 4 h + v % 4
  if (fp >= NB) return;
  const int f = lane & 31;
  if (chunks == 1) {
    // the only chunk: the rows k_bwd_finish would form from it (the same
    // operations: its sum over one partial is 0 + s = s)
    uint16_t* out = ft == 0 ? gk : gv;
    const float sc = ft == 0 ? scale : 1.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int g = fcol_group(32 * fp + 8 * (v >> 2) + 4 * h + (v & 3), nb8);
      if (g >= N) continue;
      const int cnt = count[bh * N + g];
      out[(bh * Npad + g) * 64 + f] = (uint16_t)bf16_bits(cnt > 0 ? sc * (0.f + acc0[v]) / (float)cnt : 0.f);
      out[(bh * Npad + g) * 64 + 32 + f] = (uint16_t)bf16_bits(cnt > 0 ? sc * (0.f + acc1[v]) / (float)cnt : 0.f);
    }
    return;
  }
  float* out = part + ((bh * chunks + chunk) * 2 + ft) * (int64_t)Npad * 64;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int g = fcol_group(32 * fp + 8 * (v >> 2) + 4 * h + (v & 3), nb8);
    out[g * 64 + f] = acc0[v];
    out[g * 64 + 32 + f] = acc1[v];
  }
}

// grid (Npad / 16, BH), 256 threads: thread = (group, 4 features) of 16 groups.
// gk = scale sum_chunks dr / c, gv = sum_chunks dmu / c (0 for an empty
// group), rounded to bf16 once: the rows every member key receives.
__global__ __launch_bounds__(256) void k_bwd_finish(const float* __restrict__ part, const int32_t* __restrict__ count,
                                                    int N, int Npad, int chunks, float scale, uint16_t* __restrict__ gk,
                                                    uint16_t* __restrict__ gv) {
  constexpr int kMaxC = 8;
  const int64_t bh = blockIdx.y;
  const int g = blockIdx.x * 16 + (threadIdx.x >> 4), f = 4 * (threadIdx.x & 15);
  if (g >= N) return;
  float4 sr = make_float4(0.f, 0.f, 0.f, 0.f), sm = sr;
  for (int c0 = 0; c0 < chunks; c0 += kMaxC) {
    float4 pr[kMaxC], pm[kMaxC];
#pragma unroll
    for (int c = 0; c < kMaxC; ++c) {  // up to kMaxC chunks' loads issued before their sums
      if (c0 + c < chunks) {
        const float* p = part + ((bh * chunks + c0 + c) * 2) * (int64_t)Npad * 64 + g * 64 + f;
        pr[c] = *(const float4*)p;
        pm[c] = *(const float4*)(p + (int64_t)Npad * 64);
      }
    }
#pragma unroll
    for (int c = 0; c < kMaxC; ++c) {  // in chunk order
      if (c0 + c < chunks) {
        sr.x += pr[c].x; sr.y += pr[c].y; sr.z += pr[c].z; sr.w += pr[c].w;
        sm.x += pm[c].x; sm.y += pm[c].y; sm.z += pm[c].z; sm.w += pm[c].w;
      }
    }
  }
  const int cnt = count[bh * N + g];
  const float k = (float)cnt;
  u32x2 ok = {0u, 0u}, ov = {0u, 0u};
  if (cnt > 0) {
    ok = u32x2{pack2(scale * sr.x / k, scale * sr.y / k), pack2(scale * sr.z / k, scale * sr.w / k)};
    ov = u32x2{pack2(sm.x / k, sm.y / k), pack2(sm.z / k, sm.w / k)};
  }
  *(u32x2*)(gk + (bh * Npad + g) * 64 + f) = ok;
  *(u32x2*)(gv + (bh * Npad + g) * 64 + f) = ov;
}

// grid (ceil(n / 32), BH), 256 threads: threads 0..127 write dK, 128..255 dV;
// 8 lanes per key row (16 bytes each), two keys per thread (k and k + 16),
// both keys' loads issued before the stores.
__global__ __launch_bounds__(256) void k_bwd_keys(const int32_t* __restrict__ belong, const uint16_t* __restrict__ gk,
                                                  const uint16_t* __restrict__ gv, int n, int N, int Npad,
                                                  uint16_t* __restrict__ dK, uint16_t* __restrict__ dV) {
  const int64_t bh = blockIdx.y;
  const int t = threadIdx.x & 127, which = threadIdx.x >> 7;
  const int k0 = blockIdx.x * 32 + (t >> 3), ch = t & 7;
  const uint16_t* src = which ? gv : gk;
  uint16_t* dst = which ? dV : dK;
  int g[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) g[u] = k0 + 16 * u < n ? belong[bh * n + k0 + 16 * u] : -1;
  u32x4 o[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    o[u] = u32x4{0u, 0u, 0u, 0u};
    if ((unsigned)g[u] < (unsigned)N) o[u] = *(const u32x4*)(src + (bh * Npad + g[u]) * 64 + 8 * ch);
  }
#pragma unroll
  for (int u = 0; u < 2; ++u)
    if (k0 + 16 * u < n) *(u32x4*)(dst + (bh * n + k0 + 16 * u) * 64 + 8 * ch) = o[u];
}

int bwd_npad(int N) { return (N + 31) / 32 * 32; }
int bwd_rts(int N) { return bwd_npad(N) + 4; }

}  // namespace

int backward_max_groups() { return 256; }

size_t backward_workspace_layout(const Dims& d, BackwardWorkspace* w, void* base) {
  const int Npad = bwd_npad(d.N), rts = bwd_rts(d.N);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += (bytes + 255) & ~(size_t)255;
    return base ? (char*)base + o : nullptr;
  };
  const bool fused = Npad <= 128;  // the fused kernel stages the group rows itself and keeps no statistics
  void* R = fused ? nullptr : take((size_t)d.BH * Npad * 64 * 2);
  void* RT = fused ? nullptr : take((size_t)d.BH * 64 * rts * 2);
  void* MU = fused ? nullptr : take((size_t)d.BH * Npad * 64 * 2);
  void* LC = fused ? nullptr : take((size_t)d.BH * Npad * 4);
  void* ST = fused ? nullptr : take((size_t)d.BH * d.n * 8);
  const int chunks = fused ? fused_chunks(d.BH, d.n) : bwd_chunks(d.BH, Npad / 32);
  void* PART = take((size_t)d.BH * chunks * 2 * Npad * 64 * 4);
  void* GK = take((size_t)d.BH * Npad * 64 * 2);  // bf16 rows
  void* GV = take((size_t)d.BH * Npad * 64 * 2);
  if (w) *w = BackwardWorkspace{(uint16_t*)R, (uint16_t*)RT, (uint16_t*)MU, (float*)LC, ST, (float*)PART,
                                (uint16_t*)GK, (uint16_t*)GV};
  return off;
}

hipError_t launch_backward(const Dims& d, const void* Q, const void* dO, const int32_t* belong,
                           const float* centroid, const int32_t* count, const float* vsum, float scale, void* dQ,
                           void* dK, void* dV, const BackwardWorkspace& w, hipStream_t st) {
  const int Npad = bwd_npad(d.N), rts = bwd_rts(d.N), NB = Npad / 32;
  const float sl2e = scale * 1.4426950408889634f;
  if (NB <= 4) {
    const int chunks = fused_chunks(d.BH, d.n);
    {
      TimedLaunch tl("bwd_fused", st);
#define GA_BWD_F(NBV)                                                                                              \
  hipLaunchKernelGGL(k_bwd_fused<NBV>, dim3((unsigned)(d.BH * chunks)), dim3(512), 0, st, (const uint16_t*)Q,      \
                     (const uint16_t*)dO, centroid, count, vsum, d.n, d.N, chunks, scale, sl2e, (uint16_t*)dQ,    \
                     w.part, w.gk, w.gv)
      switch (NB) {
        case 1: GA_BWD_F(1); break;
        case 2: GA_BWD_F(2); break;
        case 3: GA_BWD_F(3); break;
        default: GA_BWD_F(4); break;
      }
#undef GA_BWD_F
    }
    if (chunks > 1) {
      TimedLaunch tl("bwd_finish", st);
      hipLaunchKernelGGL(k_bwd_finish, dim3((unsigned)(Npad / 16), (unsigned)d.BH), dim3(256), 0, st, w.part, count,
                         d.N, Npad, chunks, scale, w.gk, w.gv);
    }
    TimedLaunch tl("bwd_keys", st);
    hipLaunchKernelGGL(k_bwd_keys, dim3((unsigned)((d.n + 31) / 32), (unsigned)d.BH), dim3(256), 0, st, belong,
                       w.gk, w.gv, d.n, d.N, Npad, (uint16_t*)dK, (uint16_t*)dV);
    return hipGetLastError();
  }
  {
    TimedLaunch tl("bwd_prep", st);
    hipLaunchKernelGGL(k_bwd_prep, dim3((unsigned)NB, (unsigned)d.BH), dim3(256), 0, st, centroid, count, vsum, d.N,
                       Npad, rts, w.R, w.RT, w.MU, w.LC);
  }
  const int64_t ntiles = ((int64_t)d.n + 31) / 32;
  // about one round of kBwdTargetWgs workgroups: the same number per slice
  const int64_t per_slice = (kBwdTargetWgs + d.BH - 1) / d.BH;
  const int tpw = (int)((ntiles + 4 * per_slice - 1) / (4 * per_slice));
  const unsigned gq = (unsigned)((ntiles + 4 * tpw - 1) / (4 * tpw));
  {
    TimedLaunch tl("bwd_query", st);
#define GA_BWD_Q(NBV)                                                                                              \
  hipLaunchKernelGGL(k_bwd_query<NBV>, dim3(gq, (unsigned)d.BH), dim3(256), 0, st, (const uint16_t*)Q,            \
                     (const uint16_t*)dO, w.R, w.RT, w.MU, w.LC, d.n, rts, scale, sl2e, tpw, (uint16_t*)dQ,       \
                     (float2*)w.stats)
    switch (NB) {
      case 5: GA_BWD_Q(5); break;
      case 6: GA_BWD_Q(6); break;
      case 7: GA_BWD_Q(7); break;
      default: GA_BWD_Q(8); break;
    }
#undef GA_BWD_Q
  }
  const int chunks = bwd_chunks(d.BH, NB);
  {
    TimedLaunch tl("bwd_group", st);
#define GA_BWD_G(NBV)                                                                                              \
  hipLaunchKernelGGL(k_bwd_group<NBV>, dim3((unsigned)((NBV * chunks * d.BH + 7) / 8 * 8)), dim3(256), 0, st,     \
                     (const uint16_t*)Q, (const uint16_t*)dO, w.R, w.MU, w.LC, (const float2*)w.stats, d.n, d.BH,  \
                     chunks, sl2e, w.part, count, d.N, scale, w.gk, w.gv)
    switch (NB) {
      case 5: GA_BWD_G(5); break;
      case 6: GA_BWD_G(6); break;
      case 7: GA_BWD_G(7); break;
      default: GA_BWD_G(8); break;
    }
#undef GA_BWD_G
  }
  if (chunks > 1) {  // (one chunk: k_bwd_group wrote the rows itself)
    TimedLaunch tl("bwd_finish", st);
    hipLaunchKernelGGL(k_bwd_finish, dim3((unsigned)(Npad / 16), (unsigned)d.BH), dim3(256), 0, st, w.part, count,
                       d.N, Npad, chunks, scale, w.gk, w.gv);
  }
  TimedLaunch tl("bwd_keys", st);
  hipLaunchKernelGGL(k_bwd_keys, dim3((unsigned)((d.n + 31) / 32), (unsigned)d.BH), dim3(256), 0, st, belong,
                     w.gk, w.gv, d.n, d.N, Npad, (uint16_t*)dK, (uint16_t*)dV);
  return hipGetLastError();
}

}  // namespace ga
