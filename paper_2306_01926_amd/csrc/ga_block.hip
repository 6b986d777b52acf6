// gfx950 (MI355X) projection GEMMs of the group-attention block.
//
// The RITA encoder is a Transformer encoder whose self-attention is replaced by
// group attention (Section 3); its queries, keys and values are the bias-free
// projections Q = H W_Q, K = H W_K, V = H W_V of the token embeddings (Eq. 1),
// one d = 64 slice per head, and the heads' outputs are concatenated and
// projected by W_O.  Both projections are dense contractions over
// d_model = H * 64, so they run on the matrix cores:
//
//   k_project<kQKV>  X [B, n, D] x Wqkv [3D, D]^T, written as Q, K, V
//                    [B, H, n, 64] (the layout the group-attention kernels read)
//   k_project<kOut>  O [B, H, n, 64] read head by head as the rows of
//                    [B n, D], x Wo [D, D]^T -> Y [B, n, D]
//
// bf16 operands, fp32 accumulation (MFMA 32x32x16), outputs rounded once to
// bf16 (round to nearest even).  Weights are stored one output feature per
// row ([out][in], the contraction axis contiguous).
//
// Each workgroup (4 waves) computes a tile of 256 tokens x 128 outputs over
// k-chunks of 64: the chunk's token rows and weight rows are staged in LDS
// (16-byte granules XOR-swizzled by row so that the MFMA operand reads are
// conflict-free), the next chunk's global loads are in flight during the
// MFMAs.  Each wave owns 128 tokens x 64 outputs.  The MFMA computes the
// transposed product (weights as the A operand, tokens as the B operand), and
// the weight rows feeding the A operand are permuted so that each lane ends
// with 16 consecutive output features of one token: the epilogue stores 32
// contiguous bytes per lane, straight from registers.
//
// Tiles are numbered with the output tiles of one token tile consecutive and
// handed to the XCDs in contiguous ranges (workgroup w runs on XCD w % 8), so
// the up to 12 workgroups that read the same token rows share one L2.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "ga_internal.h"

namespace ga {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kQKV = 0, kOut = 1;
constexpr int kTM = 256;  // tokens per tile
constexpr int kTO = 128;  // output features per tile
constexpr int kXBytes = kTM * 128;  // one k-chunk (64 bf16) of the token rows
constexpr int kWBytes = kTO * 128;  // one k-chunk of the weight rows

// LDS byte offset of 16-byte granule q (0..7) of row r of a token tile.  The
// granule index is XORed with a 3-bit key of the row so that the 16-byte
// reads of one MFMA operand (lane i: row i, the same granule) hit distinct
// bank groups both per 8 lanes (128 bytes) and per 16 lanes (256 bytes): the
// key takes all 8 values on 8 aligned consecutive rows, and on the even and
// on the odd rows of 16 (a 256-byte line holds an even and an odd row).
__device__ __forceinline__ int xkey(int r) { return (r & 7) ^ ((r >> 3) & 1); }
__device__ __forceinline__ int xoff(int r, int q) { return r * 128 + ((q ^ xkey(r)) << 4); }
// The weight tile is read in the order of wrow below (lane rho: row
// wrow(rho)): its key is xkey of that read rank.
__device__ __forceinline__ int wkey(int r) { return ((r & 3) | ((r >> 2) & 4)) ^ ((r >> 2) & 1); }
__device__ __forceinline__ int woff(int r, int q) { return r * 128 + ((q ^ wkey(r)) << 4); }

// Weight row (within a 32-row block) fed to MFMA row rho: output row
// rho = 8 (i / 4) + 4 h + (i % 4) of accumulator register i on lane half h
// then holds output feature 16 h + i.
__device__ __forceinline__ int wrow(int rho) { return 16 * ((rho >> 2) & 1) + 4 * (rho >> 3) + (rho & 3); }

// two values rounded to bf16 (nearest even) in one v_cvt_pk_bf16_f32
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// grid: ceil(tiles / 8) * 8 workgroups of 256 threads; tiles = tiles_m * tiles_o.
// A: kQKV: X [M][D];  kOut: O [B][H][n][64] (row m = b n + t, k-chunk = head).
// W: [Odim][D].  M = B n tokens, D = 64 H.
template <int MODE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_project(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ W, int64_t M, int n, int H, int Odim,
    int tiles_o, int64_t tiles, uint16_t* __restrict__ out0, uint16_t* __restrict__ out1,
    uint16_t* __restrict__ out2) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[kXBytes + kWBytes];
  const int64_t per = gridDim.x / 8;
  const int64_t tile = (int64_t)(blockIdx.x % 8) * per + blockIdx.x / 8;
  if (tile >= tiles) return;
  const int64_t m0 = (tile / tiles_o) * kTM;
  const int o0 = (int)(tile % tiles_o) * kTO;
  const int D = 64 * H, nk = H;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  // staging: thread tid moves granule q = tid % 8 of rows tid / 8 + 32 u
  const int q = tid & 7, r0 = tid >> 3;
  int64_t xrow[8];  // element offset of each staged token row at k-chunk 0
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const int64_t m = min(m0 + r0 + 32 * u, M - 1);
    if (MODE == kQKV) {
      xrow[u] = m * D;
    } else {
      const int64_t b = m / n, t = m - b * n;
      xrow[u] = (b * H * n + t) * 64;
    }
  }
  const int64_t xstep = MODE == kQKV ? 64 : (int64_t)n * 64;  // next k-chunk
  int64_t wrow0[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) wrow0[u] = (int64_t)min(o0 + r0 + 32 * u, Odim - 1) * D;

  u32x4 gx[8], gw[4];
  auto load = [&](int kc) {
#pragma unroll
    for (int u = 0; u < 8; ++u) gx[u] = *(const u32x4*)(A + xrow[u] + kc * xstep + 8 * q);
#pragma unroll
    for (int u = 0; u < 4; ++u) gw[u] = *(const u32x4*)(W + wrow0[u] + kc * 64 + 8 * q);
  };
  auto stage = [&]() {
#pragma unroll
    for (int u = 0; u < 8; ++u) *(u32x4*)(smem + xoff(r0 + 32 * u, q)) = gx[u];
#pragma unroll
    for (int u = 0; u < 4; ++u) *(u32x4*)(smem + kXBytes + woff(r0 + 32 * u, q)) = gw[u];
  };

  // wave tile: tokens 128 wm .. +128 (4 blocks), outputs 64 wo .. +64 (2 blocks)
  const int wm = wave & 1, wo = wave >> 1;
  const int r = lane & 31, h = lane >> 5;
  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  load(0);
  for (int kc = 0; kc < nk; ++kc) {
    stage();
    __syncthreads();
    if (kc + 1 < nk) load(kc + 1);
    // MFMA step s contracts k = 8 s .. 8 s + 7 (lane half 0) and 32 + 8 s ..
    // (half 1) of the chunk: the same permutation on both operands.
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int g = 4 * h + s;
      u32x4 fw[2], fx[4];
#pragma unroll
      for (int j = 0; j < 2; ++j)
        fw[j] = *(const u32x4*)(smem + kXBytes + woff(64 * wo + 32 * j + wrow(r), g));
#pragma unroll
      for (int i = 0; i < 4; ++i) fx[i] = *(const u32x4*)(smem + xoff(128 * wm + 32 * i + r, g));
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fw[j]),
                                                               __builtin_bit_cast(bf16x8, fx[i]), acc[i][j], 0, 0,
                                                               0);
    }
    __syncthreads();
  }

  // epilogue: lane (r, h) of block (i, j) holds outputs o .. o + 15 of token m
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t m = m0 + 128 * wm + 32 * i + r;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int o = o0 + 64 * wo + 32 * j + 16 * h;
      if (o >= Odim) continue;
      u32x4 lo, hi;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        lo[v] = pack2(acc[i][j][2 * v], acc[i][j][2 * v + 1]);
        hi[v] = pack2(acc[i][j][8 + 2 * v], acc[i][j][8 + 2 * v + 1]);
      }
      uint16_t* dst;
      if (MODE == kQKV) {
        const int which = o / D, rem = o - which * D, head = rem >> 6, c = rem & 63;
        const int64_t b = m / n, t = m - b * n;
        uint16_t* base = which == 0 ? out0 : (which == 1 ? out1 : out2);
        dst = base + ((b * H + head) * n + t) * 64 + c;
      } else {
        dst = out0 + m * Odim + o;
      }
      *(u32x4*)dst = lo;
      *(u32x4*)(dst + 8) = hi;
    }
  }
}

}  // namespace

hipError_t launch_project(int mode, int B, int n, int H, const void* A, const void* W, void* out0, void* out1,
                          void* out2, hipStream_t st) {
  const int64_t M = (int64_t)B * n;
  const int D = 64 * H;
  const int Odim = mode == 0 ? 3 * D : D;
  const int tiles_o = (Odim + kTO - 1) / kTO;
  const int64_t tiles = ((M + kTM - 1) / kTM) * tiles_o;
  const int64_t grid = (tiles + 7) / 8 * 8;
  if (mode == 0) {
    TimedLaunch tl("proj_qkv", st);
    hipLaunchKernelGGL(k_project<kQKV>, dim3((unsigned)grid), dim3(256), 0, st, (const uint16_t*)A,
                       (const uint16_t*)W, M, n, H, Odim, tiles_o, tiles, (uint16_t*)out0, (uint16_t*)out1,
                       (uint16_t*)out2);
  } else {
    TimedLaunch tl("proj_out", st);
    hipLaunchKernelGGL(k_project<kOut>, dim3((unsigned)grid), dim3(256), 0, st, (const uint16_t*)A,
                       (const uint16_t*)W, M, n, H, Odim, tiles_o, tiles, (uint16_t*)out0, nullptr, nullptr);
  }
  return hipGetLastError();
}

}  // namespace ga
