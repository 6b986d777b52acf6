// Internal interface between the C ABI (ga_abi.cpp) and the gfx950 kernels
// (ga_kernels.hip).  Every launcher enqueues on `st` and returns the
// hipError_t of the launch.
#pragma once
#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace ga {

constexpr int kD = 64;          // supported feature width
constexpr int kMaxGroups = 1024;

// Device workspace carved from the caller's buffer (all 256-byte aligned).
struct Workspace {
  float* C;          // [BH][N][64] fp32 centroids (used when the caller passes none)
  void* R;           // [BH][N][64] representatives in the storage dtype
  double* nrm64;     // [BH][N] canonical fp64 |r_j|^2
  uint16_t* nsplit;  // [BH][N][8] bf16 hi, mid, lo with hi + mid + lo ~ nrm64 (rest zero)
  float* knorm;      // [BH][n] upper bound of |k_i| (bf16 path)
  int32_t* belong;   // [BH][n]
  int32_t* perm;     // [BH][n] keys sorted by group, ascending key index inside a group
  int32_t* goff;     // [BH][N] first position of each group in perm
  int32_t* count;    // [BH][N]
  float* vsum;       // [BH][N][64]
  uint16_t* Rq;      // [BH][N][64] bf16 representatives for the scores
  uint16_t* Vt;      // [BH][64][vt_stride] bf16 per-group value means, transposed
  float* ginit;      // [BH][Npad] score-accumulator init, log2(count)/(|scale| log2 e)
  double* S64;       // [BH][N][64] fp64 member sums carried across rounds (bf16 path)
  int32_t* mcount;   // [2][BH] moved-key records of rounds t with t % 2 = 0, 1
  unsigned long long* mrec;  // [BH][n] records (key << 32 | old << 16 | new)
  double* Sp;        // [BH][kFusedP][N][64] per-partition fp64 sums of the fused update
  int32_t* cntp;     // [BH][kFusedP][N] per-partition member counts
  uint32_t* pbits;   // [BH][kFusedP][4] groups with members in each partition (bit g)
  double* lxs;       // persistent grouping (ga_lloyd.hip): [lloyd_exchange_rows(d)][64] exchanged group sums
  int32_t* lxc;      // [lloyd_exchange_rows(d)] exchanged member-count deltas
  int32_t* lxm;      // [BH][16] keys of each rank that changed group in a round
  uint32_t* lsync;   // [BH][32] barrier counters
  uint32_t* lstatus; // [64] status word (bit 0: a barrier gave up)
};

// First round of the bf16 path for N <= kFusedG: every assign workgroup (one
// partition of a slice's keys, at most kFusedP per slice) forms the initial
// representatives itself (no init launch), then sums the rows of its keys per
// group into its own partition of Sp; launch_part_finish adds the partitions
// into S64 and forms count, C, R, |r|^2 and the split.
constexpr int kFusedG = 128;
constexpr int kFusedP = 8;
struct FusedUpdate {
  double* Sp;
  int32_t* cntp;
  uint32_t* pbits;
  const float* init;  // [BH][N][64] given initial centroids, or null (strided keys)
  float* C;           // [BH][N][64] receives the initial centroids
};

struct Dims {
  int64_t BH;
  int n, N, dtype;   // dtype: 0 fp32, 1 bf16
};

// Kernel timing (see ga_timing_enable): brackets one launch with events when
// enabled on this thread.
class TimedLaunch {
 public:
  TimedLaunch(const char* name, hipStream_t st);
  ~TimedLaunch();

 private:
  int slot_;
  hipStream_t st_;
};

int vt_stride(int N);  // row stride (elements) of Vt
// Factor that widens the certification bound of the MFMA scores: GA_CERT_WIDEN
// in the environment (read at every launch), 1 to 65536, default 1.  A wider
// bound only sends more keys to the exact fp64 decision, so the results do not
// change; the tests use it to run the exact path on every key.
float cert_widen();
size_t workspace_layout(const Dims& d, Workspace* ws, void* base);  // returns bytes
// Layout of the allocation-free forward (persistent grouping + bf16 attention):
// only C, R, nrm64, nsplit, belong, count, Vt, ginit and the grouping kernel's
// lxs / lxc / lxm / lsync / lstatus are set, the rest are null.  Returns bytes.
size_t noalloc_layout(const Dims& d, Workspace* ws, void* base);

// Static scratch of the allocation-free forward (ga_noalloc.hip): a file-scope
// device array of kStaticScratchBytes per GPU, held until the process ends.
// static_scratch returns its device address on the current device (looked up
// once per device).
constexpr size_t kStaticScratchBytes = size_t(32) << 20;
hipError_t static_scratch(void** out);

hipError_t launch_init(const Dims& d, const void* K, const float* init, float* C, void* R,
                       double* nrm64, uint16_t* nsplit, int32_t* mcount, hipStream_t st);
// Partitions per slice of the first round's fused assign launch (which then
// also does the init), 0 if that launch is not used for d.
int fused_first_parts(const Dims& d);
// First round, bf16, N <= kFusedG and at most kFusedP workgroups per slice:
// the assign launch also writes the partition sums of the round's update (fu)
// and *parts is their number per slice, to be finished by launch_part_finish;
// else *parts = 0 and the caller runs the update (fu unused).
hipError_t launch_assign(const Dims& d, const void* K, const void* R, const uint16_t* nsplit,
                         const double* nrm64, float* knorm, int32_t* belong, int32_t* mcount,
                         unsigned long long* mrec, bool first, const FusedUpdate& fu, int* parts,
                         hipStream_t st);
hipError_t launch_part_finish(const Dims& d, int parts, const FusedUpdate& fu, double* S64,
                              int32_t* count, float* C, void* R, double* nrm64, uint16_t* nsplit,
                              hipStream_t st);
// bf16 path: exact fp64 group sums, each workgroup finishing its own groups (see ga_kernels.hip)
hipError_t launch_gsum(const Dims& d, int mode, const void* X, const int32_t* belong,
                       const unsigned long long* mrec, const int32_t* mcount_cur, int32_t* mcount_next,
                       double* S64, int32_t* count, float* out, void* R, double* nrm64, uint16_t* nsplit,
                       hipStream_t st);
// bf16 forward: value sums straight into the attention inputs (Vt, ginit), in
// place of launch_gsum(mode 2) + launch_attend_prep
hipError_t launch_valuesum_prep(const Dims& d, const void* V, const int32_t* belong, const int32_t* count,
                                float scale, uint16_t* Vt, float* ginit, hipStream_t st);
hipError_t launch_bucket(const Dims& d, const int32_t* belong, int32_t* perm, int32_t* goff,
                         int32_t* count, hipStream_t st);
hipError_t launch_update(const Dims& d, const void* K, const int32_t* perm, const int32_t* goff,
                         const int32_t* count, float* C, void* R, double* nrm64, uint16_t* nsplit,
                         hipStream_t st);
hipError_t launch_valuesum(const Dims& d, const void* V, const int32_t* perm,
                           const int32_t* goff, const int32_t* count, float* vsum,
                           hipStream_t st);
hipError_t launch_attend_prep(const Dims& d, const float* centroid, const int32_t* count,
                              const float* vsum, float scale, uint16_t* Rq, uint16_t* Vt,
                              float* ginit, bool make_rq, hipStream_t st);
hipError_t launch_attend(const Dims& d, const void* Q, const void* R, const uint16_t* Vt,
                         const float* ginit, const float* centroid, const int32_t* count,
                         const float* vsum, float scale, void* O, hipStream_t st);

// Persistent grouping (ga_lloyd.hip): every Lloyd round, the update and (if V
// is given) the value sums in one launch, for bf16, N <= 128 and shapes whose
// workgroups (P per slice) are all resident at once.  Writes belong, count, C,
// the final R / nsplit / nrm64 in w, and vsum and/or Vt + ginit if given.
size_t lloyd_exchange_rows(const Dims& d);  // rows (of 64 fp64) of w.lxs: B*H * (most ranks per slice) * Npad
// w.lstatus after a persistent grouping launch: kLloydMark, | 1 if a
// cross-workgroup wait gave up
constexpr uint32_t kLloydMark = 0x600d0000u;
bool lloyd_usable(const Dims& d);
int lloyd_ranks(const Dims& d);       // workgroups per slice, 0 if not usable
hipError_t launch_lloyd(const Dims& d, const void* K, const void* V, const float* init, int iters, int32_t* belong,
                        int32_t* count, float* C, const Workspace& w, float* vsum, uint16_t* Vt, float* ginit,
                        float scale, hipStream_t st);

// Projections of the attention block (ga_block.hip), bf16 with fp32
// accumulation.  mode 0: X [B][n][64H] x Wqkv[192H][64H]^T -> out0/1/2 = Q, K, V
// [B][H][n][64];  mode 1: O [B][H][n][64] x Wo[64H][64H]^T -> out0 = Y [B][n][64H].
hipError_t launch_project(int mode, int B, int n, int H, const void* A, const void* W, void* out0, void* out1,
                          void* out2, hipStream_t st);

// Merge plan of the adaptive group count (ga_merge.hip): per slice the group
// radii, the Lemma 1 threshold and the lowest S1 partner of each S2 group.
int merge_max_groups();
hipError_t launch_merge_plan(const Dims& d, const void* Q, const void* K, const int32_t* belong,
                             const float* centroid, const int32_t* count, double abs_scale, double log_eps,
                             double* radius, double* dthr, int32_t* partner, int32_t* merges, hipStream_t st);

// Backward pass (ga_backward.hip), bf16, N <= backward_max_groups().
struct BackwardWorkspace {
  uint16_t* R;   // [BH][Npad][64] bf16 representatives (R .. stats: N > 128 only)
  uint16_t* RT;  // [BH][64][Npad + 4] the same, transposed
  uint16_t* MU;  // [BH][Npad][64] bf16 value means
  float* LC;     // [BH][Npad] log2(count), -inf for an empty group
  void* stats;   // [BH][n] float2: softmax shift + log2(sum) (log2 domain), D = dO . o per query
  float* part;   // [BH][chunks][2][Npad][64] per-chunk sums of dp q and w dO
  uint16_t* gk;  // [BH][Npad][64] bf16 scale dr / count
  uint16_t* gv;  // [BH][Npad][64] bf16 dmu / count
};
int backward_max_groups();
size_t backward_workspace_layout(const Dims& d, BackwardWorkspace* w, void* base);  // returns bytes
hipError_t launch_backward(const Dims& d, const void* Q, const void* dO, const int32_t* belong,
                           const float* centroid, const int32_t* count, const float* vsum, float scale, void* dQ,
                           void* dK, void* dV, const BackwardWorkspace& w, hipStream_t st);

}  // namespace ga
