// gfx950 (MI355X): every Lloyd round of the key grouping (Section 4.4) and
// the embedding aggregation of Algorithm 1 in one launch (bf16, N <= 128).
//
// Slice bh is handled by P workgroups of 8 waves (rank r = 0 .. P-1).  Rank r
// owns the keys [r kpw, (r + 1) kpw) and the groups g = r, r + P, r + 2P, ...
// Each round (Section 4.4: assign every key to its nearest representative,
// then move every representative to the mean of its members):
//
//   1. assign: every rank scores its keys against all representatives (MFMA
//      32x32x16 bf16, packed top-2, certified argmin with the exact fp64
//      fallback; the same decision procedure as k_assign_reg) and adds the
//      rows of its keys that changed group into per-group fp64 sums in LDS
//      (joins +, leaves -): in the first round, where every key joins, straight
//      from the registers that hold the key tiles; later, in a pass over the
//      few moved keys;
//   2. every rank publishes its sums for the groups it does not own (deltas
//      of this round) and zeroes them; barrier A over the slice's P ranks;
//   3. update: every rank adds the other ranks' deltas for its groups into its
//      exact fp64 member sums, which stay in LDS for the whole launch; then
//      C = (float)(S / count) (an empty group keeps C), R = bf16(C), the
//      canonical |r|^2 and its split, published for the slice;
//   4. barrier B; every rank reads the slice's new representatives.
//
// The member sums of bf16 keys are exact in fp64 (while (e_max - e_min) +
// log2 count <= 45, see ga_kernels.hip), so the order in which the ranks and
// the LDS atomics add them cannot change a bit: groups, counts and centroids
// are those of the oracle.  A round in which no key of the slice changes group
// is a fixed point: every later round would repeat it, so the slice stops
// there with the same result.  After the last round every rank sums the value
// rows of its keys per group the same way (Algorithm 1, aggregation), the
// owners add the other ranks' parts and write the attention's inputs (bf16
// value means, transposed, and the log2(count) score bias), so the forward
// needs no other launch before the attention.
//
// Barriers: the ranks of a slice are launched on one XCD (workgroup ids
// 8 k + x all run on XCD x), all workgroups are co-resident (the host checks
// the occupancy), and every wait is bounded: past the spin limit a workgroup
// sets the status word and all workgroups leave.  Data crossing a barrier is
// written and read with device-scope (sc1) accesses, so it is coherent
// whichever XCD each rank runs on; a rank arrives only after its own stores
// have completed (s_waitcnt vmcnt(0)).
#include <hip/hip_runtime.h>

#include <float.h>
#include <math.h>
#include <stdint.h>

#include "ga_internal.h"

namespace ga {
namespace {

#include "ga_device.h"

constexpr int kLW = 8;            // waves per workgroup
constexpr int kLT = kLW * 64;     // threads per workgroup
constexpr int kLCap = 4096;       // keys per rank (LDS state)
constexpr int kLSort = 4096;      // sorted entries per pass of the sums
constexpr int kLSA = 65;          // row stride (fp64) of the LDS sums: rows of distinct groups start in distinct banks
constexpr int kLMaxWG = 256;      // workgroups of one launch at most (one per MI355X compute unit)

// The LDS sums keep feature d of a row at position pi(d) (the 8 x 8 transpose
// of the row): the eight lanes that add one 16-byte chunk of a row (features
// 8 j + f, f fixed per instruction) then hit eight distinct banks.
__host__ __device__ constexpr int lloyd_pi(int d) { return ((d & 7) << 3) | (d >> 3); }
constexpr int kLNone = 255;       // the "no group" of the first round
constexpr int kLExactB = 4;       // keys decided together by the exact fallback
constexpr uint32_t kLSpin = 1u << 22;  // polls before a barrier gives up

// ------------------------------------------------------------ device-scope access
__device__ __forceinline__ void st_dev(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev(int32_t* p, int32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev64(double* p, double v) {
  __hip_atomic_store((unsigned long long*)p, (unsigned long long)__double_as_longlong(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_dev(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int32_t ld_dev(const int32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double ld_dev64(const double* p) {
  return __longlong_as_double(
      (long long)__hip_atomic_load((const unsigned long long*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}

// The thread index through an opaque move: each phase of the round loop forms
// its addresses from it locally, so the compiler cannot hoist them out of the
// loop and keep them live across the scoring loop (whose register use would
// then spill them to scratch, and scratch reloads wait on the same counter as
// the device-scope stores).
__device__ __forceinline__ int opaque_tid() {
  int t;
  asm volatile("v_mov_b32 %0, %1" : "=v"(t) : "v"((int)threadIdx.x));
  return t;
}

// Workgroup barrier that orders LDS only: it waits for this thread's LDS
// operations (lgkmcnt), not for its global stores, so the device-scope stores
// of a phase complete in the background; the slice barrier waits for them.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

struct LloydArgs {
  const uint16_t* K;   // [BH][n][64] bf16
  const uint16_t* V;   // [BH][n][64] bf16 or null (no aggregation)
  const float* init;   // [BH][N][64] fp32 initial centroids or null (strided keys)
  int n, N, BH, P, kpw, T;
  float cm, cp;        // certification constants (see launch_lloyd)
  int32_t* belong;     // [BH][n]
  int32_t* count;      // [BH][N]
  float* C;            // [BH][N][64]
  uint16_t* R;         // [BH][N][64] representatives, exchanged every round
  uint16_t* nsplit;    // [BH][N][8]
  double* nrm64;       // [BH][N]
  double* xs;          // [BH][P][Npad][64] each rank's sums for the groups it does not own
  int32_t* xc;         // [BH][P][Npad] and the member-count deltas
  int32_t* xm;         // [BH][16] keys of each rank that changed group in the round
  uint32_t* sync;      // [BH][32] barrier counters (zero at launch)
  uint32_t* status;    // bit 0: a barrier gave up
  float* vsum;         // [BH][N][64] fp32 value sums or null
  uint16_t* Vt;        // [BH][64][vts] bf16 value means, transposed, or null
  float* ginit;        // [BH][Npad] score bias log2(count) / sl2e
  int vts;
  float inv_sl2e;
};

// LDS layout (dynamic part), in bytes from the base; Go = groups per rank.
struct LloydLds {
  double* SA;      // [Npad][kLSA] the rank's groups: exact member sums; other groups: this round's deltas
  int* dcA;        // [Npad] member-count deltas of the rank's keys
  uint16_t* Rs;    // [Npad][64] -2R, swizzled (swz)
  uint16_t* Ns;    // [Npad][8] |r|^2 split
  double* nrm;     // [Npad] canonical |r|^2
  float* knorm;    // [kLCap] |k| bounds of the rank's keys
  uint32_t* ent;   // [kLCap] moved keys from the bottom, uncertain keys from the top
  uint32_t* X;     // scratch: the exact fallback's key rows, the finished bf16 rows, the sorted entries
  uint32_t* srt;   // [kLSort] (in X) entries sorted by group: key | leave << 31
  uint8_t* eg;     // [kLSort] (in X) the entries' groups
  uint8_t* bst;    // [kLCap] the rank's keys' groups
  int* ecnt;       // [Npad] entries per group (zero between sorts)
  int* eoff;       // [Npad + 1]
  int* ecur;       // [Npad]
  int* cnt;        // [Go] member counts of the rank's groups
};

constexpr int kLRowS = 36;  // LDS row stride (words) of the finished bf16 rows
__host__ __device__ constexpr int lloyd_go(int Npad, int P) { return (Npad + P - 1) / P; }
__host__ __device__ constexpr size_t cmax(size_t x, size_t y) { return x > y ? x : y; }
__host__ __device__ constexpr size_t lloyd_x_bytes(int Npad, int P) {
  return cmax(cmax((size_t)kLW * kLExactB * 64 * 8, (size_t)lloyd_go(Npad, P) * kLRowS * 4), (size_t)kLSort * 5);
}
__host__ __device__ constexpr size_t lloyd_lds_bytes(int Npad, int P) {
  return (size_t)Npad * kLSA * 8 + (size_t)Npad * 4 + (size_t)Npad * 128 + (size_t)Npad * 16 + (size_t)Npad * 8 +
         (size_t)kLCap * 4 + (size_t)kLCap * 4 + lloyd_x_bytes(Npad, P) + (size_t)kLCap +
         (size_t)(3 * Npad + 1) * 4 + (size_t)lloyd_go(Npad, P) * 4 + 64;
}

__device__ __forceinline__ LloydLds lloyd_layout(unsigned char* base, int Npad, int P) {
  LloydLds l;
  unsigned char* p = base;
  l.SA = (double*)p;         p += (size_t)Npad * kLSA * 8;
  l.dcA = (int*)p;           p += (size_t)Npad * 4;
  l.Rs = (uint16_t*)p;       p += (size_t)Npad * 128;
  l.Ns = (uint16_t*)p;       p += (size_t)Npad * 16;
  l.nrm = (double*)p;        p += (size_t)Npad * 8;
  l.knorm = (float*)p;       p += (size_t)kLCap * 4;
  l.ent = (uint32_t*)p;      p += (size_t)kLCap * 4;
  l.X = (uint32_t*)p;        p += lloyd_x_bytes(Npad, P);
  l.srt = l.X;
  l.eg = (uint8_t*)(l.X + kLSort);
  l.bst = p;                 p += kLCap;
  l.ecnt = (int*)p;          p += (size_t)Npad * 4;
  l.eoff = (int*)p;          p += (size_t)(Npad + 1) * 4;
  l.ecur = (int*)p;          p += (size_t)Npad * 4;
  l.cnt = (int*)p;
  return l;
}

// ------------------------------------------------------------ barrier
// Arrive at barrier number k (0-based) of the slice and wait for all P ranks.
// Returns false if the wait gave up (spin limit) or another workgroup did.
__device__ __forceinline__ bool slice_barrier(uint32_t* ctr, uint32_t* status, int P, int k, int* s_flag) {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this thread's stores have completed
  __syncthreads();
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t target = (uint32_t)P * (uint32_t)(k + 1);
    int ok = 1;
    for (uint32_t spins = 0;; ++spins) {
      if (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= target) break;
      if ((spins & 255u) == 255u && (__hip_atomic_load(status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & 1u)) {
        ok = 0;
        break;
      }
      if (spins >= kLSpin) {
        __hip_atomic_fetch_or(status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    *s_flag = ok;
  }
  __syncthreads();
  return *s_flag != 0;
}

// ------------------------------------------------------------ representatives
// -2r of a bf16 pair word (exact), and the swizzled store of 16 bytes of row g.
__device__ __forceinline__ uint32_t neg2_pair(uint32_t w) {
  const uint32_t lo = __float_as_uint(bf16_to_f32(w & 0xffffu) * -2.0f) >> 16;
  const uint32_t hi = __float_as_uint(bf16_to_f32(w >> 16) * -2.0f) >> 16;
  return lo | (hi << 16);
}

// Canonical |r|^2 (fp64 fma chain over c = 0..63) of row g from the LDS copy
// of -2R (x * -0.5 is exact), its split into Ns and the value into nrm.
__device__ __forceinline__ double lds_row_norm(const LloydLds& L, int g) {
  double nrm = 0.0;
#pragma unroll
  for (int ch = 0; ch < 8; ++ch) {
    const u32x4 v = *(const u32x4*)(L.Rs + swz(g, ch));
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const double lo = (double)(-0.5f * bf16_to_f32(v[e] & 0xffffu));
      const double hi = (double)(-0.5f * bf16_to_f32(v[e] >> 16));
      nrm = fma(lo, lo, nrm);
      nrm = fma(hi, hi, nrm);
    }
  }
  return nrm;
}

// First round: every rank forms all initial representatives itself, C0_j =
// k_{floor(j n / N)} (R = C exactly) or the given init (R = bf16(C)); padded
// groups get zero rows and the largest bf16 as |r|^2 (they never win).  The
// owners write C for their groups.
__device__ void lloyd_stage_init(const LloydArgs& a, const LloydLds& L, int Npad, int64_t s, int r, double* red) {
  const int tid = threadIdx.x;
  const uint16_t* Kbh = a.K + s * (int64_t)a.n * 64;
  const float* ibh = a.init ? a.init + s * (int64_t)a.N * 64 : nullptr;
  float* Cbh = a.C + s * (int64_t)a.N * 64;
  for (int idx = tid; idx < Npad * 8; idx += kLT) {
    const int row = idx >> 3, ch = idx & 7;
    u32x4 w = {0u, 0u, 0u, 0u};
    if (row < a.N) {
      float c[8];
      if (ibh) {
        const float4 x = *(const float4*)(ibh + row * 64 + ch * 8), y = *(const float4*)(ibh + row * 64 + ch * 8 + 4);
        c[0] = x.x; c[1] = x.y; c[2] = x.z; c[3] = x.w; c[4] = y.x; c[5] = y.y; c[6] = y.z; c[7] = y.w;
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = f32_to_bf16(c[2 * e]) | (f32_to_bf16(c[2 * e + 1]) << 16);
      } else {
        w = *(const u32x4*)(Kbh + ((int64_t)row * a.n / a.N) * 64 + ch * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          c[2 * e] = bf16_to_f32(w[e] & 0xffffu);
          c[2 * e + 1] = bf16_to_f32(w[e] >> 16);
        }
      }
      if (row % a.P == r) {
        *(float4*)(Cbh + row * 64 + ch * 8) = float4{c[0], c[1], c[2], c[3]};
        *(float4*)(Cbh + row * 64 + ch * 8 + 4) = float4{c[4], c[5], c[6], c[7]};
      }
    }
    u32x4 v;
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = neg2_pair(w[e]);
    *(u32x4*)(L.Rs + swz(row, ch)) = v;
  }
  lds_barrier();
  for (int g = tid; g < Npad; g += kLT) {
    if (g < a.N) {
      const double nrm = lds_row_norm(L, g);
      L.nrm[g] = nrm;
      write_nsplit(nrm, L.Ns + g * 8);
    } else {
      L.nrm[g] = 0.0;
      *(u32x4*)(L.Ns + g * 8) = u32x4{0x7f7fu, 0u, 0u, 0u};
    }
  }
  // the largest |r|^2 (padded groups hold 0), one value per wave of groups
  if (tid < ((Npad + 63) & ~63)) {  // whole waves; lanes past Npad repeat group Npad - 1
    double m = L.nrm[min(tid, Npad - 1)];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = fmax(m, __shfl_xor(m, off));
    if ((tid & 63) == 0) red[tid >> 6] = m;
  }
}

// Later rounds: the slice's representatives published by their owners.
__device__ void lloyd_read_reps(const LloydArgs& a, const LloydLds& L, int64_t s, double* red) {
  constexpr int kU = 128 * 8 / kLT;  // 16-byte chunks of R per thread, N <= 128
  const int tid = opaque_tid();
  const uint32_t* Rw = (const uint32_t*)(a.R + s * (int64_t)a.N * 64);
  const uint32_t* Nw = (const uint32_t*)(a.nsplit + s * (int64_t)a.N * 8);
  // every load first (one round trip), clamped into the slice's rows
  u32x4 v[kU];
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int idx = min(tid + kLT * u, a.N * 8 - 1), row = idx >> 3, ch = idx & 7;
#pragma unroll
    for (int e = 0; e < 4; ++e) v[u][e] = ld_dev(Rw + row * 32 + ch * 4 + e);
  }
  const int gq = min(tid, a.N - 1);
  const uint32_t n0 = ld_dev(Nw + gq * 4), n1 = ld_dev(Nw + gq * 4 + 1);
  const double nr = ld_dev64(a.nrm64 + s * a.N + gq);
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int idx = tid + kLT * u, row = idx >> 3, ch = idx & 7;
    if (idx >= a.N * 8) continue;
    u32x4 w;
#pragma unroll
    for (int e = 0; e < 4; ++e) w[e] = neg2_pair(v[u][e]);
    *(u32x4*)(L.Rs + swz(row, ch)) = w;
  }
  if (tid < a.N) {
    *(u32x4*)(L.Ns + tid * 8) = u32x4{n0, n1, 0u, 0u};
    L.nrm[tid] = nr;
  }
  // the largest |r|^2, one value per wave of groups (threads past N hold group N - 1's)
  if (tid < ((a.N + 63) & ~63)) {
    double m = nr;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = fmax(m, __shfl_xor(m, off));
    if ((tid & 63) == 0) red[tid >> 6] = m;
  }
}

// ------------------------------------------------------------ assignment
// The certification bound of ga_kernels.hip,
//   E = (cm Mk + cp (|M1| + 3 cm Mk)) (1 + 2^-20) + 2^-22 |M1| + 1e-30,
//   Mk = nmax + 2 |k| rmax,
// regrouped as eA + eB |k| + eC |M1| with the per-round uniform terms formed
// once (equal in real arithmetic; the few extra fp32 roundings are far inside
// the 2^-20 margin).
struct LloydCert {
  float eA, eB, eC;
};
__device__ __forceinline__ LloydCert lloyd_cert(float nmaxf, float rmaxf, float cm, float cp) {
  const float f = 1.0f + 0x1p-20f, cmm = cm * (1.0f + 3.0f * cp);
  LloydCert c;
  c.eA = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(cmm * nmaxf * f + 1e-30f)));
  c.eB = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(2.0f * cmm * rmaxf * f)));
  c.eC = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(cp * f + 0x1p-22f)));
  return c;
}

// Decision for the keys of two tiles A and B (see decide_pair in
// ga_kernels.hip for the lane swap): certain keys get their group in bst and,
// after the first round, a moved-key entry from the bottom of ent if it
// changed; uncertain keys are queued from the top of ent for the exact
// fallback.
__device__ __forceinline__ void lloyd_decide(float M1a, float M2a, int B1a, float M1b, float M2b, int B1b, float knv,
                                             int oldv, int lk, bool valid, bool first, int N, const LloydCert& cf,
                                             const LloydLds& L, int* s_nmov, int* s_nunc) {
  const auto p1 = __builtin_amdgcn_permlane32_swap(__float_as_uint(M1a), __float_as_uint(M1b), false, false);
  const auto p2 = __builtin_amdgcn_permlane32_swap(__float_as_uint(M2a), __float_as_uint(M2b), false, false);
  const auto pb = __builtin_amdgcn_permlane32_swap((uint32_t)B1a, (uint32_t)B1b, false, false);
  const float a1 = __uint_as_float(p1[0]), b1 = __uint_as_float(p1[1]);
  const bool hi_wins = b1 < a1;
  const uint32_t vw = __float_as_uint(hi_wins ? b1 : a1) & kPackMask;
  const int jstar = 32 * (int)(hi_wins ? pb[1] : pb[0]) + 8 * (int)(vw >> 2) + (hi_wins ? 4 : 0) + (int)(vw & 3);
  const float best = min2(a1, b1);
  const float second = min2(max2(a1, b1), min2(__uint_as_float(p2[0]), __uint_as_float(p2[1])));
  const float E = fmaf(fabsf(best), cf.eC, knv * cf.eB) + cf.eA;
  const bool certain = (second > fmaf(2.0f, E, best)) && (jstar < N);
  if (valid && certain) L.bst[lk] = (uint8_t)jstar;
  const bool mv = valid && certain && !first && jstar != oldv;
  const bool un = valid && !certain;
  const uint64_t mm = __ballot(mv), mu = __ballot(un);
  const int lane = threadIdx.x & 63;
  int bm = 0, bu = 0;
  if (lane == 0) {
    if (mm) bm = atomicAdd(s_nmov, (int)__popcll(mm));
    if (mu) bu = atomicAdd(s_nunc, (int)__popcll(mu));
  }
  bm = __builtin_amdgcn_readlane(bm, 0);
  bu = __builtin_amdgcn_readlane(bu, 0);
  const uint64_t below = (1ull << lane) - 1ull;
  if (mv) L.ent[bm + (int)__popcll(mm & below)] = (uint32_t)lk | ((uint32_t)oldv << 12) | ((uint32_t)jstar << 20);
  if (un) L.ent[kLCap - 1 - (bu + (int)__popcll(mu & below))] = (uint32_t)lk | ((uint32_t)oldv << 12);
}

template <int NB>
__device__ __forceinline__ void lloyd_assign(const LloydArgs& a, const LloydLds& L, int64_t s, int k0, int nk,
                                             bool first, bool rev, const LloydCert& cf, int* s_nmov, int* s_nunc) {
  const int tid = opaque_tid();
  const int lane = tid & 63, h = lane >> 5, q = lane & 31;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ntl = (nk + 31) >> 5;
  const int tc = wv < ntl ? (ntl - wv + kLW - 1) / kLW : 0;
  const uint16_t* Kbh = a.K + s * (int64_t)a.n * 64;
  u32x4 af[NB][4], an[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    an[b] = *(const u32x4*)(L.Ns + (b * 32 + q) * 8);
#pragma unroll
    for (int s2 = 0; s2 < 4; ++s2) af[b][s2] = *(const u32x4*)(L.Rs + swz(b * 32 + q, 4 * h + s2));
  }
  const u32x4 ones = h == 0 ? u32x4{0x3f803f80u, 0x3f80u, 0u, 0u} : u32x4{0u, 0u, 0u, 0u};
  f32x16 nacc[NB];
  norm_terms<NB>(an, ones, nacc);
  if (tc == 0) return;
  // tile of the wave's j-th step: waves take every kLW-th tile, in ascending
  // order or (rev) descending, so that a round starts on the keys the previous
  // round read last
  auto tile = [&](int j) __attribute__((always_inline)) { return rev ? ntl - 1 - wv - kLW * j : wv + kLW * j; };
  // key row of tile j (wave-local index) for this lane: clamped into the slice
  auto load = [&](int j, u32x4 (&f)[4]) __attribute__((always_inline)) {
    const int key = min(k0 + tile(j) * 32 + q, a.n - 1);
    const uint16_t* krow = Kbh + (int64_t)key * 64 + h * 32;
#pragma unroll
    for (int s2 = 0; s2 < 4; ++s2) f[s2] = *(const u32x4*)(krow + s2 * 8);
  };
  auto state = [&](int j, const u32x4 (&f)[4], float& knv, int& oldv) __attribute__((always_inline)) {
    const int lk = tile(j) * 32 + q;
    if (first) {
      knv = key_norm_bound(f);
      if (h == 0 && lk < kLCap) L.knorm[lk] = knv;
      oldv = kLNone;
    } else {
      const int lkc = min(lk, kLCap - 1);
      knv = L.knorm[lkc];
      oldv = L.bst[lkc];
    }
  };
  u32x4 kb[2][4];
  load(0, kb[0]);
  for (int j = 0; j < tc; j += 2) {
    float M1a, M2a, M1b, M2b, kna, knb;
    int B1a, B1b, olda, oldb;
    load(min(j + 1, tc - 1), kb[1]);
    __builtin_amdgcn_sched_barrier(0);
    state(j, kb[0], kna, olda);
    score_tile<NB, true>(af, an, ones, nacc, kb[0], M1a, M2a, B1a);
    load(min(j + 2, tc - 1), kb[0]);
    __builtin_amdgcn_sched_barrier(0);
    const int jb = min(j + 1, tc - 1);  // past the last tile: a repeat, not decided
    state(jb, kb[1], knb, oldb);
    score_tile<NB, true>(af, an, ones, nacc, kb[1], M1b, M2b, B1b);
    // lanes h = 0 decide key q of tile j, lanes h = 1 key q of tile j + 1
    const bool valid = j + h < tc && tile(j + h) * 32 + q < nk;
    const int lk = valid ? tile(j + h) * 32 + q : 0;
    lloyd_decide(M1a, M2a, B1a, M1b, M2b, B1b, h ? knb : kna, h ? oldb : olda, lk, valid, first, a.N, cf, L, s_nmov,
                 s_nunc);
  }
}

// Exact fallback for the uncertain keys (queued from the top of ent): the
// wave takes kLExactB keys at a time and decides them in fp64; after the
// first round it adds the rows of those that changed group (fp64, from the
// LDS copy) into the sums.  The keys are dealt from the last wave down (the
// moved-key sums, which may run beside this phase, are dealt from wave 0 up).
__device__ void lloyd_exact(const LloydArgs& a, const LloydLds& L, int64_t s, int k0, int nunc, bool first,
                            int* s_xmov) {
  const int otid = opaque_tid(), lane = otid & 63;
  const int wave = kLW - 1 - __builtin_amdgcn_readfirstlane(otid >> 6);
  const uint16_t* Kbh = a.K + s * (int64_t)a.n * 64;
  double* kd = (double*)L.X + wave * kLExactB * 64;
  const int per = (nunc + kLW - 1) / kLW;
  const int u_end = min(nunc, (wave + 1) * per);
  int moved = 0;
  for (int u0 = wave * per; u0 < u_end; u0 += kLExactB) {
    const int nb = min(kLExactB, u_end - u0);
    uint32_t e[kLExactB];
#pragma unroll
    for (int b = 0; b < kLExactB; ++b) {
      e[b] = b < nb ? L.ent[kLCap - 1 - (u0 + b)] : 0u;
      if (b < nb) kd[b * 64 + lane] = (double)bf16_to_f32(Kbh[(int64_t)(k0 + (e[b] & 4095u)) * 64 + lane]);
    }
    int jb[kLExactB];
    switch (nb) {
      case 1: exact_argmin_keys<1>(kd, L.Rs, L.nrm, a.N, jb); break;
      case 2: exact_argmin_keys<2>(kd, L.Rs, L.nrm, a.N, jb); break;
      case 3: exact_argmin_keys<3>(kd, L.Rs, L.nrm, a.N, jb); break;
      default: exact_argmin_keys<4>(kd, L.Rs, L.nrm, a.N, jb); break;
    }
#pragma unroll
    for (int b = 0; b < kLExactB; ++b) {
      if (b >= nb) break;
      const int lk = (int)(e[b] & 4095u), old = (int)((e[b] >> 12) & 255u), nw = jb[b];
      if (nw == old) continue;
      if (lane == 0) L.bst[lk] = (uint8_t)nw;
      if (first) continue;  // the first round's sums are formed from every key afterwards
      const double x = kd[b * 64 + lane];
      atomicAdd(L.SA + nw * kLSA + lloyd_pi(lane), x);
      atomicAdd(L.SA + old * kLSA + lloyd_pi(lane), -x);
      if (lane == 0) {
        atomicAdd(&L.dcA[nw], 1);
        atomicAdd(&L.dcA[old], -1);
      }
      ++moved;
    }
  }
  if (lane == 0 && moved) atomicAdd(s_xmov, moved);
}

// ------------------------------------------------------------ sums
// The rows of a group-sorted entry list (srt: key | leave << 31, eg: group,
// keys local to the rank, rows from Xr) added into the LDS sums by the
// workgroup's 64 slots of 8 lanes: a slot's contiguous range is summed in
// fp64 registers while the group stays the same and flushed into the sums
// with LDS atomics when it changes (the sums are exact, so neither the cut
// nor the order matters).
constexpr int kLRunU = 8;
__device__ __forceinline__ void lloyd_run_sums(const LloydLds& L, int ne, const uint16_t* __restrict__ Xr) {
  if (ne <= 0) return;
  const int otid = opaque_tid(), lane = otid & 63, wave = __builtin_amdgcn_readfirstlane(otid >> 6);
  const int j = lane & 7, gsl = 8 * wave + (lane >> 3);
  constexpr int kSlots = 8 * kLW;
  const int b0 = (int)((int64_t)gsl * ne / kSlots), b1 = (int)((int64_t)(gsl + 1) * ne / kSlots);
  const int steps = (ne + kSlots - 1) / kSlots;
  double x[8] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
  int cur = -1;
  auto load = [&](int k0, uint32_t (&ei)[kLRunU], int (&gi)[kLRunU], u32x4 (&w)[kLRunU]) {
#pragma unroll
    for (int u = 0; u < kLRunU; ++u) {
      const int e = min(b0 + k0 + u, ne - 1);
      ei[u] = L.srt[e];
      gi[u] = L.eg[e];
      w[u] = *(const u32x4*)(Xr + (int64_t)(ei[u] & 0x7fffffffu) * 64 + 8 * j);
    }
  };
  auto flush = [&]() {
    double* p = L.SA + cur * kLSA + j;
#pragma unroll
    for (int f = 0; f < 8; ++f) {  // feature 8 j + f at position 8 f + j
      atomicAdd(p + 8 * f, x[f]);
      x[f] = 0.0;
    }
  };
  auto add = [&](int k0, const uint32_t (&ei)[kLRunU], const int (&gi)[kLRunU], const u32x4 (&w)[kLRunU]) {
#pragma unroll
    for (int u = 0; u < kLRunU; ++u) {
      if (b0 + k0 + u >= b1) break;
      if (gi[u] != cur) {
        if (cur >= 0) flush();
        cur = gi[u];
      }
      const double sg = (ei[u] >> 31) ? -1.0 : 1.0;
#pragma unroll
      for (int f = 0; f < 8; ++f)
        x[f] = fma(sg, (double)bf16_to_f32((w[u][f >> 1] >> (16 * (f & 1))) & 0xffffu), x[f]);
    }
  };
  uint32_t eA[kLRunU], eB[kLRunU];
  int gA[kLRunU], gB[kLRunU];
  u32x4 wA[kLRunU], wB[kLRunU];
  load(0, eA, gA, wA);
  for (int k0 = 0; k0 < steps; k0 += 2 * kLRunU) {
    if (k0 + kLRunU < steps) load(k0 + kLRunU, eB, gB, wB);
    add(k0, eA, gA, wA);
    if (k0 + kLRunU >= steps) break;
    if (k0 + 2 * kLRunU < steps) load(k0 + 2 * kLRunU, eA, gA, wA);
    add(k0 + kLRunU, eB, gB, wB);
  }
  if (cur >= 0) flush();
}

// Counting sort of up to kLSort entries into srt/eg by group (the counters
// ecnt must be zero), given each thread's candidate entries (gv < 0: none).
template <int PER>
__device__ __forceinline__ int lloyd_sort(const LloydLds& L, int Npad, const uint32_t (&ev)[PER],
                                          const int (&gv)[PER]) {
  const int tid = opaque_tid(), lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
#pragma unroll
  for (int u = 0; u < PER; ++u)
    if (gv[u] >= 0) atomicAdd(&L.ecnt[gv[u]], 1);
  lds_barrier();
  if (wave == 0) {  // exclusive scan over Npad <= 128 groups, two per lane
    const int ga = 2 * lane, gb = ga + 1;
    const int ca = ga < Npad ? L.ecnt[ga] : 0, cb = gb < Npad ? L.ecnt[gb] : 0;
    int incl = ca + cb;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int y = __shfl_up(incl, off);
      if (lane >= off) incl += y;
    }
    const int sa = incl - ca - cb;
    if (ga < Npad) L.eoff[ga] = L.ecur[ga] = sa;
    if (gb < Npad) L.eoff[gb] = L.ecur[gb] = sa + ca;
    if (lane == 63) L.eoff[Npad] = incl;
  }
  lds_barrier();
#pragma unroll
  for (int u = 0; u < PER; ++u)
    if (gv[u] >= 0) {
      const int pos = atomicAdd(&L.ecur[gv[u]], 1);
      L.srt[pos] = ev[u];
      L.eg[pos] = (uint8_t)gv[u];
    }
  lds_barrier();
  const int ne = L.eoff[Npad];
  if (tid < Npad) L.ecnt[tid] = 0;
  return ne;
}

// The rows of X (the keys in the first round, the values for the
// aggregation) of all the rank's keys added into the sums of their groups
// (from bst), with the member counts if `counts`.
__device__ void lloyd_sums_all(const uint16_t* X, const LloydArgs& a, const LloydLds& L, int64_t s, int k0, int nk,
                               int Npad, bool counts) {
  const int tid = opaque_tid();
  constexpr int PER = kLSort / kLT;
  uint32_t ev[PER];
  int gv[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int i = tid + kLT * u;
    ev[u] = (uint32_t)i;
    gv[u] = i < nk ? (int)L.bst[i] : -1;
    if (counts && gv[u] >= 0) atomicAdd(&L.dcA[gv[u]], 1);
  }
  const int ne = lloyd_sort<PER>(L, Npad, ev, gv);
  lloyd_run_sums(L, ne, X + (s * (int64_t)a.n + k0) * 64);
  lds_barrier();
}

// Later rounds: the rows of the rank's certain keys that changed group (from
// the bottom of ent) added into the sums, joins + and leaves -.  Up to kLDirect
// keys go straight to LDS atomics (eight lanes per row, every row loaded
// before any is added: one round trip, no sort); more are sorted by group and
// summed in registers first.
constexpr int kLPU = 4;                    // rows per lane group in the direct path
constexpr int kLDirect = kLW * 8 * kLPU;  // moved keys the direct path takes
__device__ void lloyd_sums_moved(const LloydArgs& a, const LloydLds& L, int64_t s, int k0, int nmov, int Npad) {
  const int tid = opaque_tid();
  if (nmov <= kLDirect) {
    const int lane = tid & 63, wave = tid >> 6, j = lane & 7, sub = lane >> 3;
    const uint16_t* Kr = a.K + (s * (int64_t)a.n + k0) * 64;
    uint32_t e[kLPU];
    u32x4 w[kLPU];
#pragma unroll
    for (int u = 0; u < kLPU; ++u) {
      const int i = min(wave * 8 * kLPU + 8 * u + sub, nmov - 1);  // clamped: in the list, rows in bounds
      e[u] = L.ent[i];
      w[u] = *(const u32x4*)(Kr + (int64_t)(e[u] & 4095u) * 64 + 8 * j);
    }
#pragma unroll
    for (int u = 0; u < kLPU; ++u) {
      if (wave * 8 * kLPU + 8 * u + sub >= nmov) break;
      const int old = (int)((e[u] >> 12) & 255u), nw = (int)(e[u] >> 20);
      double* pn = L.SA + nw * kLSA + j;
      double* po = L.SA + old * kLSA + j;
#pragma unroll
      for (int f = 0; f < 8; ++f) {  // feature 8 j + f at position 8 f + j
        const double x = (double)bf16_to_f32((w[u][f >> 1] >> (16 * (f & 1))) & 0xffffu);
        atomicAdd(pn + 8 * f, x);
        atomicAdd(po + 8 * f, -x);
      }
      if (j == 0) {
        atomicAdd(&L.dcA[nw], 1);
        atomicAdd(&L.dcA[old], -1);
      }
    }
    lds_barrier();
    return;
  }
  constexpr int PER = kLSort / 2 / kLT;  // moved keys per thread and pass (two entries each)
  for (int c0 = 0; c0 < nmov; c0 += kLSort / 2) {
    uint32_t ev[2 * PER];
    int gv[2 * PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int i = c0 + tid + kLT * u;
      gv[2 * u] = gv[2 * u + 1] = -1;
      ev[2 * u] = ev[2 * u + 1] = 0u;
      if (i < nmov) {
        const uint32_t e = L.ent[i];
        const int lk = (int)(e & 4095u), old = (int)((e >> 12) & 255u), nw = (int)(e >> 20);
        gv[2 * u] = nw;
        ev[2 * u] = (uint32_t)lk;
        gv[2 * u + 1] = old;
        ev[2 * u + 1] = (uint32_t)lk | 0x80000000u;
        atomicAdd(&L.dcA[nw], 1);
        atomicAdd(&L.dcA[old], -1);
      }
    }
    const int ne = lloyd_sort<2 * PER>(L, Npad, ev, gv);
    lloyd_run_sums(L, ne, a.K + (s * (int64_t)a.n + k0) * 64);
    lds_barrier();
  }
}

// ------------------------------------------------------------ exchange
// The rank's sums and count deltas for the groups it does not own go to its
// slot of the exchange buffer, and are zeroed for the next round.  Those
// groups are enumerated directly (the m-th in ascending order is member
// m mod (P-1) of block m / (P-1), skipping member r), one row per wave and
// step, kLPubB rows per wave read from LDS before any is stored.
constexpr int kLPubB = 2;
__device__ void lloyd_publish(const LloydArgs& a, const LloydLds& L, int64_t s, int r) {
  if (a.P == 1) return;
  const int tid = opaque_tid(), lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int Npad = (a.N + 31) & ~31;
  double* xs = a.xs + (s * a.P + r) * (int64_t)Npad * 64;
  int32_t* xc = a.xc + (s * a.P + r) * (int64_t)Npad;
  const int Pm = a.P - 1, Gn = a.N - (r < a.N ? (a.N - 1 - r) / a.P + 1 : 0);
  auto other = [&](int m) __attribute__((always_inline)) {
    const int i = m % Pm;
    return (m / Pm) * a.P + i + (i >= r ? 1 : 0);
  };
  for (int m0 = wave; m0 < Gn; m0 += kLW * kLPubB) {
    double v[kLPubB];
    int at[kLPubB];
#pragma unroll
    for (int b = 0; b < kLPubB; ++b) {
      const int m = m0 + kLW * b;  // wave-uniform
      at[b] = m < Gn ? other(m) : -1;
      v[b] = L.SA[max(at[b], 0) * kLSA + lane];
    }
#pragma unroll
    for (int b = 0; b < kLPubB; ++b) {
      if (at[b] < 0) break;
      st_dev64(xs + at[b] * 64 + lane, v[b]);
      L.SA[at[b] * kLSA + lane] = 0.0;
    }
  }
  for (int m = tid; m < Gn; m += kLT) {
    const int g = other(m);
    st_dev(xc + g, L.dcA[g]);
    L.dcA[g] = 0;
  }
}

// After barrier A: the other ranks' sums (and count deltas) for the rank's
// groups added into its exact sums (and counts).  The thread's (item, other
// rank) pairs are loaded kLGB at a time, all of a batch before any is added;
// the count deltas (group lg = tid mod 128 of other ranks tid / 128 + 4 k)
// and, with `want_moved`, every rank's count of keys that changed group (the
// slice's total is returned) are requested with the first batch, so that a
// slice with few ranks needs one round trip.  Every load address is clamped
// into the slice's buffers; loads past the end are not used.
constexpr int kLGB = 8;  // loads in flight per thread
__device__ __forceinline__ int lloyd_gather(const LloydArgs& a, const LloydLds& L, int64_t s, int r, int Go,
                                            bool counts, bool want_moved) {
  const int tid = opaque_tid(), lane = tid & 63;
  const int Npad = (a.N + 31) & ~31;
  const int U = (Go * 64 + kLT - 1) / kLT;  // items of this thread (some past Go * 64)
  const int pairs = U * (a.P - 1);
  const double* xs = a.xs + s * a.P * (int64_t)Npad * 64;
  int u = 0, q0 = 0;  // pair p = q0 U + u: item u of other rank q0 (ranks past r shifted by one)
  double v[kLGB];
  int at[kLGB];  // LDS position of the item, -1 past the end (the items are the thread's own: no atomics)
  auto issue = [&](int p0) __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < kLGB; ++b) {
      const int q = min(q0 + (q0 >= r), a.P - 1);
      const int idx = tid + kLT * u, lg = idx >> 6, c = idx & 63;
      const int g = min(r + a.P * min(lg, Go - 1), a.N - 1);
      at[b] = p0 + b < pairs && lg < Go && r + a.P * lg < a.N ? g * kLSA + c : -1;
      v[b] = ld_dev64(xs + ((int64_t)q * Npad + g) * 64 + c);
      if (++u == U) {
        u = 0;
        q0 = min(q0 + 1, a.P - 2);
      }
    }
  };
  auto add = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < kLGB; ++b)
      if (at[b] >= 0) L.SA[at[b]] += v[b];
  };
  if (pairs > 0) issue(0);
  const int xmv = want_moved ? ld_dev(a.xm + s * 16 + min(lane & 15, a.P - 1)) : 0;
  constexpr int kCK = 4;  // other ranks per thread for the count deltas (P <= 16)
  int cdel[kCK], cg[kCK];
  const int clg = tid & 127, cg0 = r + a.P * clg;
#pragma unroll
  for (int k = 0; k < kCK; ++k) {
    const int qo = (tid >> 7) + 4 * k, q = min(qo + (qo >= r), a.P - 1);
    cdel[k] = counts && a.P > 1 ? ld_dev(a.xc + (s * a.P + q) * (int64_t)Npad + min(cg0, a.N - 1)) : 0;
    cg[k] = counts && qo < a.P - 1 && clg < Go && cg0 < a.N ? cg0 : -1;
  }
  if (pairs > 0) add();
  for (int p0 = kLGB; p0 < pairs; p0 += kLGB) {
    issue(p0);
    add();
  }
  int moved = 1;
  if (want_moved) {  // every 16 lanes sum the P ranks' counts
    int m = (lane & 15) < a.P ? xmv : 0;
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) m += __shfl_xor(m, off);
    moved = __builtin_amdgcn_readfirstlane(m);
  }
  if (!counts) return moved;
#pragma unroll
  for (int k = 0; k < kCK; ++k)
    if (cg[k] >= 0) atomicAdd(&L.dcA[cg[k]], cdel[k]);
  lds_barrier();
  for (int lg = tid; lg < Go; lg += kLT) {
    const int g = r + a.P * lg;
    if (g >= a.N) continue;
    L.cnt[lg] += L.dcA[g];
    L.dcA[g] = 0;
  }
  return moved;
}

// ------------------------------------------------------------ update
// Finish the rank's groups after an update: C (an empty group keeps C),
// R = bf16(C), |r|^2 and its split, published for the slice; the counts too
// in the last round.
//
// The previous C of every item (prev) is loaded before barrier A,
// unconditionally: its round trip overlaps the wait, and loads and stores
// share one counter (vmcnt): a load the compiler cannot track (e.g. a
// conditional one) would make it wait for every earlier store, including the
// slow device-scope ones, before each later use.
//
// |r|^2: the canonical value is the fp64 fma chain over c = 0..63.  Each
// square of a bf16 component is exact in fp64 (16 significant bits); if the
// nonzero squares of a row span at most 31 binades, every partial sum in any
// order is a multiple of the smallest square's last bit and below 2^53 of it,
// so every partial sum is exact and any summation order gives the chain's
// bits (eight lanes per row sum eight squares each, then a shuffle tree).
// Rows outside that range take the chain itself.
constexpr int kLFinU = 128 * 32 / kLT;  // (group, feature pair) items per thread, Go <= 128
__device__ __forceinline__ int sq_exp(double x) {  // biased exponent of a square (0 for 0)
  return (int)((__double_as_longlong(x) >> 52) & 2047);
}
// The previous C of the rank's groups, (group, feature pair) items
// tid + kLT u (clamped loads: every address is in bounds).
__device__ __forceinline__ void lloyd_prev_c(const LloydArgs& a, int64_t s, int r, int Go, float2 (&prev)[kLFinU]) {
  const int tid = opaque_tid();
  const float* Cbh = a.C + s * (int64_t)a.N * 64;
#pragma unroll
  for (int u = 0; u < kLFinU; ++u) {
    const int idx = tid + kLT * u, lg = idx >> 5, c2 = idx & 31;
    const int g = min(r + a.P * min(lg, Go - 1), a.N - 1);
    prev[u] = *(const float2*)(Cbh + g * 64 + 2 * c2);
  }
}

__device__ void lloyd_finish(const LloydArgs& a, const LloydLds& L, int64_t s, int r, int Go, bool last,
                             float2 (&prev)[kLFinU]) {
  const int tid = opaque_tid();
  float* Cbh = a.C + s * (int64_t)a.N * 64;
  uint32_t* Rw = (uint32_t*)(a.R + s * (int64_t)a.N * 64);
  uint32_t* rows = L.X;  // [Go][kLRowS] bf16 pairs
#pragma unroll
  for (int u = 0; u < kLFinU; ++u) {
    const int idx = tid + kLT * u, lg = idx >> 5, c2 = idx & 31, g = r + a.P * lg;
    if (lg >= Go || g >= a.N) continue;
    const int cnt = L.cnt[lg];
    float c0 = prev[u].x, c1 = prev[u].y;
    if (cnt > 0) {
      c0 = (float)(L.SA[g * kLSA + lloyd_pi(2 * c2)] / (double)cnt);
      c1 = (float)(L.SA[g * kLSA + lloyd_pi(2 * c2 + 1)] / (double)cnt);
    }
    prev[u] = float2{c0, c1};
    rows[lg * kLRowS + c2] = f32_to_bf16(c0) | (f32_to_bf16(c1) << 16);
  }
  lds_barrier();
  // per group (eight lanes, eight features each): |r|^2, its split, the count
  for (int base = 0; base < Go * 8; base += kLT) {
    const int t = base + tid, lg = t >> 3, j = t & 7, g = r + a.P * lg;
    const bool ok = lg < Go && g < a.N;
    const u32x4 w = ok ? *(const u32x4*)(rows + lg * kLRowS + 4 * j) : u32x4{0u, 0u, 0u, 0u};
    double acc = 0.0;
    int emax = 0, emin = 4096;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t bits = (e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xffffu);
      const double rc = (double)bf16_to_f32(bits);
      const double q = rc * rc;  // exact
      acc += q;
      if (q != 0.0) {
        emax = max(emax, sq_exp(q));
        emin = min(emin, sq_exp(q));
      }
    }
#pragma unroll
    for (int off = 1; off < 8; off <<= 1) {  // the group's eight lanes are consecutive lanes of one wave
      acc += __shfl_xor(acc, off);
      emax = max(emax, __shfl_xor(emax, off));
      emin = min(emin, __shfl_xor(emin, off));
    }
    if (!ok || j != 0) continue;
    double nrm = acc;
    if (emin != 4096 && emax - emin > 31) {  // not provably exact: the chain itself
      nrm = 0.0;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const u32x4 wk = *(const u32x4*)(rows + lg * kLRowS + 4 * k);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const double rc = (double)bf16_to_f32((e & 1) ? (wk[e >> 1] >> 16) : (wk[e >> 1] & 0xffffu));
          nrm = fma(rc, rc, nrm);
        }
      }
    }
    uint16_t sp[8];
    write_nsplit(nrm, sp);
    uint32_t* Nw = (uint32_t*)(a.nsplit + (s * a.N + g) * 8);
    st_dev(Nw, (uint32_t)sp[0] | ((uint32_t)sp[1] << 16));
    st_dev(Nw + 1, (uint32_t)sp[2] | ((uint32_t)sp[3] << 16));
    st_dev64(a.nrm64 + s * a.N + g, nrm);
    if (last) a.count[s * a.N + g] = L.cnt[lg];
  }
  // C (non-empty groups) and R
#pragma unroll
  for (int u = 0; u < kLFinU; ++u) {
    const int idx = tid + kLT * u, lg = idx >> 5, c2 = idx & 31, g = r + a.P * lg;
    if (lg >= Go || g >= a.N) continue;
    if (L.cnt[lg] > 0) *(float2*)(Cbh + g * 64 + 2 * c2) = prev[u];
    st_dev(Rw + g * 32 + c2, f32_to_bf16(prev[u].x) | (f32_to_bf16(prev[u].y) << 16));
  }
  lds_barrier();
}

// ------------------------------------------------------------ aggregation
// Outputs of the aggregation for the rank's groups (and the attention's padded
// groups up to a multiple of 32): vsum = (float) of the exact sum, the bf16
// means transposed (Vt) and the score bias log2(count) / (|scale| log2 e).
__device__ void lloyd_value_outputs(const LloydArgs& a, const LloydLds& L, int64_t s, int r, int Go) {
  const int tid = opaque_tid();
  const int NpA = (a.N + 31) & ~31;
  for (int idx = tid; idx < Go * 64; idx += kLT) {
    const int lg = idx >> 6, c = idx & 63, g = r + a.P * lg;
    if (g >= NpA) continue;
    const bool real = g < a.N;
    const float vs = real ? (float)L.SA[g * kLSA + lloyd_pi(c)] : 0.f;
    const int cnt = real ? L.cnt[lg] : 0;
    if (a.vsum && real) a.vsum[(s * a.N + g) * 64 + c] = vs;
    if (a.Vt) {
      a.Vt[(s * 64 + c) * (int64_t)a.vts + g] = (uint16_t)f32_to_bf16(cnt > 0 ? vs / (float)cnt : 0.f);
      if (c == 0) a.ginit[s * NpA + g] = cnt > 0 ? log2f((float)cnt) * a.inv_sl2e : -INFINITY;
    }
  }
}

// ------------------------------------------------------------ kernel
template <int NB>
__global__ __launch_bounds__(kLT) void k_lloyd(LloydArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int s_nmov, s_nunc, s_xmov, s_flag;
  __shared__ double s_red[kLW];
  constexpr int Npad = NB * 32;
  const int tid = threadIdx.x;
  const int bx = blockIdx.x, idx = bx >> 3;
  const int64_t s = (int64_t)(idx / a.P) * 8 + (bx & 7);
  const int r = idx % a.P;
  if (s >= a.BH) return;
  const int Go = lloyd_go(Npad, a.P);
  const LloydLds L = lloyd_layout(smem, Npad, a.P);
  const int k0 = r * a.kpw, nk = max(0, min(a.kpw, a.n - k0));
  uint32_t* ctr = a.sync + s * 32;
  int bar = 0;

  if (tid == 0) {  // the round's key counters (cleared again after each barrier A)
    s_nmov = 0;
    s_nunc = 0;
    s_xmov = 0;
  }
  lloyd_stage_init(a, L, Npad, s, r, s_red);
  for (int i = tid; i < Npad * kLSA; i += kLT) L.SA[i] = 0.0;
  for (int i = tid; i < Npad; i += kLT) {
    L.dcA[i] = 0;
    L.ecnt[i] = 0;
  }
  for (int i = tid; i < Go; i += kLT) L.cnt[i] = 0;
  lds_barrier();

  for (int t = 0; t < a.T; ++t) {
    const bool first = t == 0;
    bool last = t == a.T - 1;
    // certification constants from the largest |r|^2 of the slice (one value
    // per wave of groups, left by lloyd_stage_init / lloyd_read_reps)
    double nmax = s_red[0];
    if (Npad > 64) nmax = fmax(nmax, s_red[1]);
    const float nmaxf = (float)nmax * (1.0f + 0x1p-20f);
    const LloydCert cf = lloyd_cert(nmaxf, sqrtf(nmaxf) * (1.0f + 0x1p-20f), a.cm, a.cp);

    // 1. assignment of the rank's keys and the sums of those that changed group
    lloyd_assign<NB>(a, L, s, k0, nk, first, (t & 1) != 0, cf, &s_nmov, &s_nunc);
    lds_barrier();
    const int nunc = s_nunc, nmov = s_nmov;
    // after the first round, with few moved keys (their sums take the direct
    // path, which uses no LDS scratch), the exact fallback and the moved-key
    // sums run side by side: both add exact values into the sums
    const bool side = !first && nmov <= kLDirect;
    if (nunc) {
      lloyd_exact(a, L, s, k0, nunc, first, &s_xmov);
      if (!side || nmov == 0) lds_barrier();
    }
    if (first)  // every key joins its group
      lloyd_sums_all(a.K, a, L, s, k0, nk, Npad, true);
    else if (nmov)
      lloyd_sums_moved(a, L, s, k0, nmov, Npad);
    // 2. the deltas of the other ranks' groups, then barrier A
    lloyd_publish(a, L, s, r);
    if (tid == 0) st_dev(a.xm + s * 16 + r, first ? nk : nmov + s_xmov);
    float2 prev[kLFinU];
    lloyd_prev_c(a, s, r, Go, prev);
    if (!slice_barrier(ctr, a.status, a.P, bar++, &s_flag)) return;
    if (tid == 0) {  // every use of this round's key counters is behind the barrier
      s_nmov = 0;
      s_nunc = 0;
      s_xmov = 0;
    }
    // 3. update of the rank's groups; a round in which no key of the slice
    // changed group is a fixed point, so it is the last
    if (lloyd_gather(a, L, s, r, Go, true, !first && !last) == 0) last = true;
    lds_barrier();
    lloyd_finish(a, L, s, r, Go, last, prev);
    if (last) break;
    // 4. barrier B, then the slice's new representatives
    if (!slice_barrier(ctr, a.status, a.P, bar++, &s_flag)) return;
    lloyd_read_reps(a, L, s, s_red);
    lds_barrier();
  }
  // the groups of the rank's keys
  for (int i = tid; i < nk; i += kLT) a.belong[s * (int64_t)a.n + k0 + i] = (int32_t)L.bst[i];
  if (!a.V) return;
  // aggregation: value sums of the rank's keys per group, exchanged like the
  // key sums (barrier B first: every rank has read the last round's deltas)
  for (int i = tid; i < Npad * kLSA; i += kLT) L.SA[i] = 0.0;
  lds_barrier();
  lloyd_sums_all(a.V, a, L, s, k0, nk, Npad, false);
  if (!slice_barrier(ctr, a.status, a.P, bar++, &s_flag)) return;
  lloyd_publish(a, L, s, r);
  if (!slice_barrier(ctr, a.status, a.P, bar++, &s_flag)) return;
  lloyd_gather(a, L, s, r, Go, false, false);
  lds_barrier();
  lloyd_value_outputs(a, L, s, r, Go);
}

// Clears the barrier counters and marks the status word as belonging to a
// persistent grouping launch (kLloydMark, failure bit 0 clear).
__global__ void k_lloyd_reset(uint32_t* sync, int words, uint32_t* status) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < words; i += gridDim.x * blockDim.x) sync[i] = 0u;
  if (blockIdx.x == 0 && threadIdx.x == 0) *status = kLloydMark;
}

}  // namespace
}  // namespace ga

// ------------------------------------------------------------ host side
#include <map>
#include <mutex>
#include <tuple>

namespace ga {
namespace {

using LloydFn = void (*)(LloydArgs);
const LloydFn kLloydFns[4] = {k_lloyd<1>, k_lloyd<2>, k_lloyd<3>, k_lloyd<4>};

// Most ranks per slice: about one per 256 keys, at most 16, and at most
// kLMaxWG workgroups in the launch (this also bounds the exchange buffer,
// whose size must not depend on the device).
int lloyd_pcap(const Dims& d) {
  const int64_t bh8x8 = (std::max<int64_t>(d.BH, 1) + 7) / 8 * 8;
  const int64_t p = std::min<int64_t>(std::min<int64_t>(16, ((int64_t)d.n + 255) / 256), kLMaxWG / bh8x8);
  return (int)std::max<int64_t>(1, p);
}

// Compute units of the current device and the workgroups of `fn` (512
// threads, `lds` bytes of dynamic LDS) each holds at once; cached.
std::pair<int, int> lloyd_capacity(int nb, size_t lds) {
  static std::mutex mu;
  static std::map<std::tuple<int, int, size_t>, std::pair<int, int>> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return {0, 0};
  std::lock_guard<std::mutex> lock(mu);
  const auto key = std::make_tuple(dev, nb, lds);
  auto it = cache.find(key);
  if (it != cache.end()) return it->second;
  int cus = 0, occ = 0;
  const void* fn = (const void*)kLloydFns[nb - 1];
  (void)hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lloyd_lds_bytes(32 * nb, 1));
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, fn, kLT, lds) != hipSuccess) {
    (void)hipGetLastError();
    cus = occ = 0;
  }
  return cache[key] = {cus, occ};
}

struct LloydPlan {
  bool ok = false;
  int nb = 0, P = 0, kpw = 0;
  unsigned grid = 0;
  size_t lds = 0;
};

LloydPlan plan_lloyd(const Dims& d) {
  LloydPlan p;
  if (d.dtype != 1 || d.N > 128 || d.n > 65536 || d.BH < 1 || d.BH > 4096) return p;
  p.nb = (d.N + 31) / 32;
  const int Npad = 32 * p.nb;
  const int64_t bh8 = (d.BH + 7) / 8;
  // ranks per slice: about one per 256 keys, at most 16, and every workgroup
  // of the launch resident at once
  int P = lloyd_pcap(d);
  for (; P >= 1; --P) {
    const size_t lds = lloyd_lds_bytes(Npad, P);
    const auto cap = lloyd_capacity(p.nb, lds);
    if ((int64_t)bh8 * 8 * P <= (int64_t)cap.first * cap.second) {
      p.lds = lds;
      break;
    }
  }
  if (P < 1) return p;
  p.P = P;
  p.kpw = (int)(((int64_t)d.n + 32 * P - 1) / (32 * P)) * 32;
  if (p.kpw > kLCap) return p;
  p.grid = (unsigned)(bh8 * 8 * P);
  p.ok = true;
  return p;
}

}  // namespace

size_t lloyd_exchange_rows(const Dims& d) {
  return (size_t)d.BH * (size_t)lloyd_pcap(d) * (size_t)((d.N + 31) & ~31);
}

bool lloyd_usable(const Dims& d) { return plan_lloyd(d).ok; }

int lloyd_ranks(const Dims& d) {
  const LloydPlan p = plan_lloyd(d);
  return p.ok ? p.P : 0;
}

hipError_t launch_lloyd(const Dims& d, const void* K, const void* V, const float* init, int iters, int32_t* belong,
                        int32_t* count, float* C, const Workspace& w, float* vsum, uint16_t* Vt, float* ginit,
                        float scale, hipStream_t st) {
  const LloydPlan p = plan_lloyd(d);
  if (!p.ok) return hipErrorInvalidValue;
  {
    TimedLaunch timed("lloyd_reset", st);
    const int words = (int)(d.BH * 32);
    hipLaunchKernelGGL(k_lloyd_reset, dim3((unsigned)std::min(64, (words + 255) / 256)), dim3(256), 0, st, w.lsync,
                       words, w.lstatus);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  TimedLaunch timed("lloyd", st);
  LloydArgs a{};
  a.K = (const uint16_t*)K;
  a.V = (const uint16_t*)V;
  a.init = init;
  a.n = d.n;
  a.N = d.N;
  a.BH = (int)d.BH;
  a.P = p.P;
  a.kpw = p.kpw;
  a.T = iters;
  // certification constants: see launch_assign (MFMA accumulation error and
  // the 4 packed index bits)
  a.cm = (float)(kD + 4) * 0x1p-23f * (1.0f + 0x1p-10f) * cert_widen();
  a.cp = 0x1p-19f * (1.0f + 0x1p-10f) * cert_widen();
  a.belong = belong;
  a.count = count;
  a.C = C;
  a.R = (uint16_t*)w.R;
  a.nsplit = w.nsplit;
  a.nrm64 = w.nrm64;
  a.xs = w.lxs;
  a.xc = w.lxc;
  a.xm = w.lxm;
  a.sync = w.lsync;
  a.status = w.lstatus;
  a.vsum = vsum;
  a.Vt = Vt;
  a.ginit = ginit;
  a.vts = vt_stride(d.N);
  const float sl2e = std::max(fabsf(scale) * 1.4426950408889634f, 1e-30f);
  a.inv_sl2e = 1.0f / sl2e;
  hipLaunchKernelGGL(kLloydFns[p.nb - 1], dim3(p.grid), dim3(kLT), p.lds, st, a);
  return hipGetLastError();
}

}  // namespace ga
