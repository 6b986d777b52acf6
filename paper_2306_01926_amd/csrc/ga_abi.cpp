// C ABI of libga.so (declared in include/ga.h): argument validation on the
// host, workspace carve-up and the launch sequence of each entry point.
#include "ga.h"

#include <hip/hip_runtime_api.h>

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <string>
#include <vector>

#include "ga_internal.h"

float ga::cert_widen() {
  const char* e = getenv("GA_CERT_WIDEN");
  if (!e) return 1.0f;
  char* end = nullptr;
  const double v = strtod(e, &end);
  return end != e && v >= 1.0 && v <= 65536.0 ? (float)v : 1.0f;
}

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(GA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Shape checks shared by every entry point.  *empty is set for B == 0 or H == 0.
int check_shape(const ga_shape_t& s, int32_t N, bool* empty) {
  *empty = false;
  if (s.dtype != GA_F32 && s.dtype != GA_BF16) return fail(GA_ERR_INVALID_ARG, "unknown dtype %d", s.dtype);
  if (s.B < 0 || s.H < 0) return fail(GA_ERR_INVALID_ARG, "negative batch/head count (B=%d, H=%d)", s.B, s.H);
  if (s.n < 1) return fail(GA_ERR_INVALID_ARG, "n must be >= 1 (got %d)", s.n);
  if (s.d != ga::kD) return fail(GA_ERR_UNSUPPORTED, "only d = 64 is supported (got %d)", s.d);
  if (N < 1 || N > s.n || N > ga::kMaxGroups)
    return fail(GA_ERR_INVALID_ARG, "N must satisfy 1 <= N <= min(n, %d) (N=%d, n=%d)", ga::kMaxGroups, N, s.n);
  const int64_t BH = (int64_t)s.B * s.H;
  if (BH > 65535) return fail(GA_ERR_UNSUPPORTED, "B*H = %lld exceeds 65535", (long long)BH);
  if (s.n > (1 << 30)) return fail(GA_ERR_UNSUPPORTED, "n = %d too large", s.n);
  *empty = BH == 0;
  return GA_OK;
}

int check_ptr(const void* p, const char* name, bool required) {
  if (!p) return required ? fail(GA_ERR_INVALID_ARG, "%s is NULL", name) : GA_OK;
  if (!aligned16(p)) return fail(GA_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  return GA_OK;
}

int check_ws(const ga::Dims& d, void* ws, size_t bytes, ga::Workspace* w) {
  const size_t need = ga::workspace_layout(d, nullptr, nullptr);
  if (!ws) return fail(GA_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (((uintptr_t)ws & 255u) != 0) return fail(GA_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  if (bytes < need) return fail(GA_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", bytes, need);
  ga::workspace_layout(d, w, ws);
  return GA_OK;
}

ga::Dims dims_of(const ga_shape_t& s, int32_t N) {
  return ga::Dims{(int64_t)s.B * s.H, s.n, N, s.dtype};
}

#define GA_TRY(expr)              \
  do {                            \
    const int rc_ = (expr);       \
    if (rc_ != GA_OK) return rc_; \
  } while (0)

#define GA_LAUNCH(expr, what)                     \
  do {                                            \
    const hipError_t e_ = (expr);                 \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

// Grouping on validated arguments.
// bf16: the first round sums every member; later rounds apply only the keys
// that changed group (exact fp64 sums make the order irrelevant), with a
// group-sum launch over round t's moved-key records, counted in mcount[t % 2].
// For N <= kFusedG with few enough assign workgroups per slice the first
// round's assign launch writes per-workgroup partition sums and a small launch
// adds them.  fp32: every round re-sums the members in ascending key order
// (fp32 sums need not be exact).
// The persistent grouping kernel (every round in one launch) serves bf16
// shapes it supports; GA_GROUPING=rounds in the environment selects the
// launch-per-round path instead (for comparisons).
bool use_persistent(const ga::Dims& d) {
  const char* e = getenv("GA_GROUPING");
  if (e && strcmp(e, "rounds") == 0) return false;
  return d.dtype == GA_BF16 && ga::lloyd_usable(d);
}

int run_cluster(const ga::Dims& d, const void* K, int32_t iters, const float* init, int32_t* belong,
                int32_t* count, float* C, const ga::Workspace& w, hipStream_t st) {
  if (use_persistent(d)) {
    GA_LAUNCH(ga::launch_lloyd(d, K, nullptr, init, iters, belong, count, C, w, nullptr, nullptr, nullptr, 1.0f, st),
              "grouping launch");
    return GA_OK;
  }
  // with the fused first round the assign launch forms the initial centroids itself
  if (ga::fused_first_parts(d) == 0)
    GA_LAUNCH(ga::launch_init(d, K, init, C, w.R, w.nrm64, w.nsplit, w.mcount, st), "init launch");
  const ga::FusedUpdate fu{w.Sp, w.cntp, w.pbits, init, C};
  for (int t = 0; t < iters; ++t) {
    int32_t* mc_cur = w.mcount + (t & 1) * d.BH;
    int32_t* mc_next = w.mcount + ((t + 1) & 1) * d.BH;
    int parts = 0;
    GA_LAUNCH(ga::launch_assign(d, K, w.R, w.nsplit, w.nrm64, w.knorm, belong, mc_cur, w.mrec, t == 0, fu, &parts,
                                st), "assign launch");
    if (parts > 0) {
      GA_LAUNCH(ga::launch_part_finish(d, parts, fu, w.S64, count, C, w.R, w.nrm64, w.nsplit, st), "update launch");
    } else if (d.dtype == GA_BF16) {
      GA_LAUNCH(ga::launch_gsum(d, t == 0 ? 0 : 1, K, belong, w.mrec, mc_cur, mc_next, w.S64, count, C, w.R,
                                w.nrm64, w.nsplit, st), "update launch");
    } else {
      GA_LAUNCH(ga::launch_bucket(d, belong, w.perm, w.goff, count, st), "bucket launch");
      GA_LAUNCH(ga::launch_update(d, K, w.perm, w.goff, count, C, w.R, w.nrm64, w.nsplit, st), "update launch");
    }
  }
  return GA_OK;
}

// Value sums for the current assignment.
int run_valuesum(const ga::Dims& d, const void* V, const int32_t* belong, int32_t* count, float* vsum,
                 const ga::Workspace& w, hipStream_t st) {
  if (d.dtype == GA_BF16) {
    GA_LAUNCH(ga::launch_gsum(d, 2, V, belong, nullptr, nullptr, nullptr, nullptr, nullptr, vsum, nullptr, nullptr,
                              nullptr, st), "value-sum launch");
  } else {
    GA_LAUNCH(ga::launch_bucket(d, belong, w.perm, w.goff, count, st), "bucket launch");
    GA_LAUNCH(ga::launch_valuesum(d, V, w.perm, w.goff, count, vsum, st), "value-sum launch");
  }
  return GA_OK;
}

// Whole forward through the persistent grouping kernel: grouping, update and
// value sums (straight into the attention's inputs) in one launch, then the
// attention.  Uses w.R, nrm64, nsplit, Vt, ginit, lxs, lxc, lxm, lsync, lstatus.
int run_forward_persistent(const ga::Dims& d, const void* Q, const void* K, const void* V, int32_t iters,
                           float scale, void* O, int32_t* belong, int32_t* count, float* C, const ga::Workspace& w,
                           hipStream_t st) {
  GA_LAUNCH(ga::launch_lloyd(d, K, V, nullptr, iters, belong, count, C, w, nullptr, w.Vt, w.ginit, scale, st),
            "grouping launch");
  GA_LAUNCH(ga::launch_attend(d, Q, w.R, w.Vt, w.ginit, C, count, nullptr, scale, O, st), "attention launch");
  return GA_OK;
}

// Whole forward on validated arguments (belong / count / centroid may be NULL).
int run_forward(const ga::Dims& d, const void* Q, const void* K, const void* V, int32_t iters, float scale, void* O,
                int32_t* belong, int32_t* count, float* centroid, const ga::Workspace& w, hipStream_t st) {
  int32_t* a = belong ? belong : w.belong;
  int32_t* cnt = count ? count : w.count;
  float* C = centroid ? centroid : w.C;
  if (use_persistent(d)) return run_forward_persistent(d, Q, K, V, iters, scale, O, a, cnt, C, w, st);
  GA_TRY(run_cluster(d, K, iters, nullptr, a, cnt, C, w, st));
  if (d.dtype == GA_BF16) {
    // the value sums go straight into the attention's transposed means and bias
    GA_LAUNCH(ga::launch_valuesum_prep(d, V, a, cnt, scale, w.Vt, w.ginit, st), "value-sum launch");
    GA_LAUNCH(ga::launch_attend(d, Q, w.R, w.Vt, w.ginit, C, cnt, w.vsum, scale, O, st), "attention launch");
  } else {
    // the last stable bucket pass sorted the keys by the final assignment: reuse it
    GA_LAUNCH(ga::launch_valuesum(d, V, w.perm, w.goff, cnt, w.vsum, st), "value-sum launch");
    GA_LAUNCH(ga::launch_attend(d, Q, nullptr, nullptr, nullptr, C, cnt, w.vsum, scale, O, st),
              "attention launch");
  }
  return GA_OK;
}

// Shape checks of the attention block (bf16 only, d = 64, d_model = 64 H <= 4096).
// with_groups: also check N against n and the bf16 attention limit.
int check_block_shape(const ga_shape_t& s, int32_t N, bool with_groups, bool* empty) {
  *empty = false;
  if (s.dtype != GA_BF16 && s.dtype != GA_F32) return fail(GA_ERR_INVALID_ARG, "unknown dtype %d", s.dtype);
  if (s.dtype != GA_BF16) return fail(GA_ERR_UNSUPPORTED, "the attention block is bf16 only");
  if (s.B < 0 || s.H < 0) return fail(GA_ERR_INVALID_ARG, "negative batch/head count (B=%d, H=%d)", s.B, s.H);
  if (s.n < 1) return fail(GA_ERR_INVALID_ARG, "n must be >= 1 (got %d)", s.n);
  if (s.d != ga::kD) return fail(GA_ERR_UNSUPPORTED, "only d = 64 is supported (got %d)", s.d);
  if (s.H > 64) return fail(GA_ERR_UNSUPPORTED, "d_model = 64 H must be <= 4096 (H=%d)", s.H);
  if ((int64_t)s.B * s.H > 65535) return fail(GA_ERR_UNSUPPORTED, "B*H exceeds 65535");
  if (s.n > (1 << 30)) return fail(GA_ERR_UNSUPPORTED, "n = %d too large", s.n);
  if (with_groups) {
    if (N < 1 || N > s.n || N > 256)
      return fail(N > 256 && N <= s.n ? GA_ERR_UNSUPPORTED : GA_ERR_INVALID_ARG,
                  "N must satisfy 1 <= N <= min(n, 256) (N=%d, n=%d)", N, s.n);
  }
  *empty = s.B == 0 || s.H == 0;
  return GA_OK;
}

// Block workspace: Q, K, V, O [B][H][n][64] bf16, then the group-attention
// workspace.  Returns the bytes; with base set, fills qkvo and w.
size_t block_ws_layout(const ga_shape_t& s, int32_t N, void* base, void** qkvo, ga::Workspace* w) {
  const size_t t = ((size_t)s.B * s.H * s.n * 64 * 2 + 255) & ~(size_t)255;
  const ga::Dims d = dims_of(s, N);
  const size_t rest = ga::workspace_layout(d, nullptr, nullptr);
  if (base) {
    for (int i = 0; i < 4; ++i) qkvo[i] = (char*)base + i * t;
    ga::workspace_layout(d, w, (char*)base + 4 * t);
  }
  return 4 * t + rest;
}

// ---------------------------------------------------------------- kernel timing
struct TimingRec {
  const char* name;
  hipEvent_t start, stop;
};
struct TimingState {
  bool on = false;
  std::vector<TimingRec> recs;
  std::vector<hipEvent_t> pool;
  hipEvent_t take() {
    hipEvent_t e = nullptr;
    if (!pool.empty()) {
      e = pool.back();
      pool.pop_back();
    } else if (hipEventCreate(&e) != hipSuccess) {
      e = nullptr;
    }
    return e;
  }
};
thread_local TimingState g_timing;

}  // namespace

namespace ga {

TimedLaunch::TimedLaunch(const char* name, hipStream_t st) : slot_(-1), st_(st) {
  if (!g_timing.on) return;
  TimingRec r{name, g_timing.take(), g_timing.take()};
  if (!r.start || !r.stop) return;
  (void)hipEventRecord(r.start, st);
  slot_ = (int)g_timing.recs.size();
  g_timing.recs.push_back(r);
}

TimedLaunch::~TimedLaunch() {
  if (slot_ >= 0) (void)hipEventRecord(g_timing.recs[slot_].stop, st_);
}

}  // namespace ga

extern "C" {

int ga_timing_enable(int on) {
  g_timing.on = on != 0;
  return GA_OK;
}

int ga_timing_collect(ga_kernel_time_t* out, int32_t max_entries, int32_t* n_entries) {
  std::vector<ga_kernel_time_t> acc;
  int status = GA_OK;
  for (const TimingRec& r : g_timing.recs) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(r.stop);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.start, r.stop);
    if (e != hipSuccess && status == GA_OK) status = hip_fail(e, "timing event");
    size_t k = 0;
    while (k < acc.size() && strncmp(acc[k].name, r.name, sizeof acc[k].name) != 0) ++k;
    if (k == acc.size()) {
      ga_kernel_time_t t{};
      snprintf(t.name, sizeof t.name, "%s", r.name);
      acc.push_back(t);
    }
    acc[k].launches += 1;
    acc[k].total_ms += ms;
    g_timing.pool.push_back(r.start);
    g_timing.pool.push_back(r.stop);
  }
  g_timing.recs.clear();
  const int32_t m = (int32_t)acc.size() < max_entries ? (int32_t)acc.size() : max_entries;
  for (int32_t i = 0; i < m; ++i) out[i] = acc[i];
  if (n_entries) *n_entries = m;
  return status;
}

size_t ga_workspace_bytes(ga_shape_t s, int32_t N) {
  bool empty;
  const std::string keep = g_last_error;
  if (check_shape(s, N, &empty) != GA_OK) {
    g_last_error = keep;
    return 0;
  }
  return ga::workspace_layout(dims_of(s, N), nullptr, nullptr);
}

int ga_workspace_check(ga_shape_t s, int32_t N, const void* workspace, size_t workspace_bytes, void* stream) {
  bool empty;
  GA_TRY(check_shape(s, N, &empty));
  if (empty) return GA_OK;
  const ga::Dims d = dims_of(s, N);
  ga::Workspace w;
  GA_TRY(check_ws(d, (void*)workspace, workspace_bytes, &w));
  GA_LAUNCH(hipStreamSynchronize((hipStream_t)stream), "stream synchronisation");
  uint32_t status = 0;
  GA_LAUNCH(hipMemcpy(&status, w.lstatus, sizeof status, hipMemcpyDeviceToHost), "status read");
  // a workspace that no persistent grouping launch used holds no status
  if ((status & 0xffff0000u) == ga::kLloydMark && (status & 1u))
    return fail(GA_ERR_HIP, "a cross-workgroup wait of the grouping launch gave up (status 0x%x): its outputs are invalid",
                status);
  return GA_OK;
}

int ga_cluster(ga_shape_t s, const void* K, int32_t N, int32_t iters, const float* init, int32_t* belong,
               int32_t* count, float* centroid, void* workspace, size_t workspace_bytes, void* stream) {
  bool empty;
  GA_TRY(check_shape(s, N, &empty));
  if (iters < 1) return fail(GA_ERR_INVALID_ARG, "iters must be >= 1 (got %d)", iters);
  GA_TRY(check_ptr(K, "K", true));
  GA_TRY(check_ptr(init, "init", false));
  GA_TRY(check_ptr(belong, "belong", true));
  GA_TRY(check_ptr(count, "count", true));
  GA_TRY(check_ptr(centroid, "centroid", true));
  if (empty) return GA_OK;
  const ga::Dims d = dims_of(s, N);
  ga::Workspace w;
  GA_TRY(check_ws(d, workspace, workspace_bytes, &w));
  return run_cluster(d, K, iters, init, belong, count, centroid, w, (hipStream_t)stream);
}

int ga_aggregate(ga_shape_t s, const void* V, const int32_t* belong, int32_t N, float* vsum, void* workspace,
                 size_t workspace_bytes, void* stream) {
  bool empty;
  GA_TRY(check_shape(s, N, &empty));
  GA_TRY(check_ptr(V, "V", true));
  GA_TRY(check_ptr(belong, "belong", true));
  GA_TRY(check_ptr(vsum, "vsum", true));
  if (empty) return GA_OK;
  const ga::Dims d = dims_of(s, N);
  ga::Workspace w;
  GA_TRY(check_ws(d, workspace, workspace_bytes, &w));
  return run_valuesum(d, V, belong, w.count, vsum, w, (hipStream_t)stream);
}

int ga_attend(ga_shape_t s, const void* Q, const float* centroid, const int32_t* count, const float* vsum,
              int32_t N, float scale, void* O, void* workspace, size_t workspace_bytes, void* stream) {
  bool empty;
  GA_TRY(check_shape(s, N, &empty));
  if (!isfinite(scale)) return fail(GA_ERR_INVALID_ARG, "scale must be finite");
  GA_TRY(check_ptr(Q, "Q", true));
  GA_TRY(check_ptr(centroid, "centroid", true));
  GA_TRY(check_ptr(count, "count", true));
  GA_TRY(check_ptr(vsum, "vsum", true));
  GA_TRY(check_ptr(O, "O", true));
  if (s.dtype == GA_BF16 && N > 256)
    return fail(GA_ERR_UNSUPPORTED, "bf16 attention supports N <= 256 (got %d)", N);
  if (empty) return GA_OK;
  const ga::Dims d = dims_of(s, N);
  ga::Workspace w;
  GA_TRY(check_ws(d, workspace, workspace_bytes, &w));
  hipStream_t st = (hipStream_t)stream;
  if (s.dtype == GA_BF16) {
    GA_LAUNCH(ga::launch_attend_prep(d, centroid, count, vsum, scale, w.Rq, w.Vt, w.ginit, true, st),
              "attention prep launch");
    GA_LAUNCH(ga::launch_attend(d, Q, w.Rq, w.Vt, w.ginit, centroid, count, vsum, scale, O, st),
              "attention launch");
  } else {
    GA_LAUNCH(ga::launch_attend(d, Q, nullptr, nullptr, nullptr, centroid, count, vsum, scale, O, st),
              "attention launch");
  }
  return GA_OK;
}

int ga_forward(ga_shape_t s, const void* Q, const void* K, const void* V, int32_t N, int32_t iters,
               float scale, void* O, int32_t* belong, int32_t* count, float* centroid, void* workspace,
               size_t workspace_bytes, void* stream) {
  bool empty;
  GA_TRY(check_shape(s, N, &empty));
  if (iters < 1) return fail(GA_ERR_INVALID_ARG, "iters must be >= 1 (got %d)", iters);
  if (!isfinite(scale)) return fail(GA_ERR_INVALID_ARG, "scale must be finite");
  GA_TRY(check_ptr(Q, "Q", true));
  GA_TRY(check_ptr(K, "K", true));
  GA_TRY(check_ptr(V, "V", true));
  GA_TRY(check_ptr(O, "O", true));
  GA_TRY(check_ptr(belong, "belong", false));
  GA_TRY(check_ptr(count, "count", false));
  GA_TRY(check_ptr(centroid, "centroid", false));
  if (s.dtype == GA_BF16 && N > 256)
    return fail(GA_ERR_UNSUPPORTED, "bf16 attention supports N <= 256 (got %d)", N);
  if (empty) return GA_OK;
  const ga::Dims d = dims_of(s, N);
  ga::Workspace w;
  GA_TRY(check_ws(d, workspace, workspace_bytes, &w));
  return run_forward(d, Q, K, V, iters, scale, O, belong, count, centroid, w, (hipStream_t)stream);
}

static_assert(GA_NOALLOC_SCRATCH_BYTES == ga::kStaticScratchBytes, "static scratch size");

int ga_forward_noalloc(ga_shape_t s, const void* Q, const void* K, const void* V, int32_t N, int32_t iters,
                       float scale, void* O, int32_t* belong, int32_t* count, float* centroid, void* stream) {
  bool empty;
  GA_TRY(check_shape(s, N, &empty));
  if (iters < 1) return fail(GA_ERR_INVALID_ARG, "iters must be >= 1 (got %d)", iters);
  if (!isfinite(scale)) return fail(GA_ERR_INVALID_ARG, "scale must be finite");
  GA_TRY(check_ptr(Q, "Q", true));
  GA_TRY(check_ptr(K, "K", true));
  GA_TRY(check_ptr(V, "V", true));
  GA_TRY(check_ptr(O, "O", true));
  GA_TRY(check_ptr(belong, "belong", false));
  GA_TRY(check_ptr(count, "count", false));
  GA_TRY(check_ptr(centroid, "centroid", false));
  if (s.dtype != GA_BF16) return fail(GA_ERR_UNSUPPORTED, "ga_forward_noalloc supports bf16 only");
  if (empty) return GA_OK;
  const ga::Dims d = dims_of(s, N);
  const size_t need = ga::noalloc_layout(d, nullptr, nullptr);
  if (need > ga::kStaticScratchBytes)
    return fail(GA_ERR_WORKSPACE, "this shape needs %zu bytes of scratch, the static scratch holds %zu", need,
                ga::kStaticScratchBytes);
  if (!ga::lloyd_usable(d))
    return fail(GA_ERR_UNSUPPORTED,
                "ga_forward_noalloc serves the one-launch grouping only: N <= 128, n <= 65536 and every workgroup "
                "of the launch resident at once (B*H=%lld, n=%d, N=%d)", (long long)d.BH, d.n, d.N);
  void* base = nullptr;
  const hipError_t e = ga::static_scratch(&base);
  if (e != hipSuccess) return hip_fail(e, "static scratch lookup");
  ga::Workspace w;
  ga::noalloc_layout(d, &w, base);
  return run_forward_persistent(d, Q, K, V, iters, scale, O, belong ? belong : w.belong, count ? count : w.count,
                                centroid ? centroid : w.C, w, (hipStream_t)stream);
}

size_t ga_block_workspace_bytes(ga_shape_t s, int32_t N) {
  bool empty;
  const std::string keep = g_last_error;
  const int rc = check_block_shape(s, N, true, &empty);
  g_last_error = keep;
  if (rc != GA_OK) return 0;
  return block_ws_layout(s, N, nullptr, nullptr, nullptr);
}

int ga_project_qkv(ga_shape_t s, const void* X, const void* Wqkv, void* Q, void* K, void* V, void* stream) {
  bool empty;
  GA_TRY(check_block_shape(s, 1, false, &empty));
  GA_TRY(check_ptr(X, "X", true));
  GA_TRY(check_ptr(Wqkv, "Wqkv", true));
  GA_TRY(check_ptr(Q, "Q", true));
  GA_TRY(check_ptr(K, "K", true));
  GA_TRY(check_ptr(V, "V", true));
  if (empty) return GA_OK;
  GA_LAUNCH(ga::launch_project(0, s.B, s.n, s.H, X, Wqkv, Q, K, V, (hipStream_t)stream), "projection launch");
  return GA_OK;
}

int ga_project_out(ga_shape_t s, const void* O, const void* Wo, void* Y, void* stream) {
  bool empty;
  GA_TRY(check_block_shape(s, 1, false, &empty));
  GA_TRY(check_ptr(O, "O", true));
  GA_TRY(check_ptr(Wo, "Wo", true));
  GA_TRY(check_ptr(Y, "Y", true));
  if (empty) return GA_OK;
  GA_LAUNCH(ga::launch_project(1, s.B, s.n, s.H, O, Wo, Y, nullptr, nullptr, (hipStream_t)stream),
            "projection launch");
  return GA_OK;
}

int ga_attention_block(ga_shape_t s, const void* X, const void* Wqkv, const void* Wo, int32_t N, int32_t iters,
                       float scale, void* Y, void* workspace, size_t workspace_bytes, void* stream) {
  bool empty;
  GA_TRY(check_block_shape(s, N, true, &empty));
  if (iters < 1) return fail(GA_ERR_INVALID_ARG, "iters must be >= 1 (got %d)", iters);
  if (!isfinite(scale)) return fail(GA_ERR_INVALID_ARG, "scale must be finite");
  GA_TRY(check_ptr(X, "X", true));
  GA_TRY(check_ptr(Wqkv, "Wqkv", true));
  GA_TRY(check_ptr(Wo, "Wo", true));
  GA_TRY(check_ptr(Y, "Y", true));
  if (empty) return GA_OK;
  const size_t need = block_ws_layout(s, N, nullptr, nullptr, nullptr);
  if (!workspace) return fail(GA_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (((uintptr_t)workspace & 255u) != 0) return fail(GA_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  if (workspace_bytes < need)
    return fail(GA_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", workspace_bytes, need);
  void* qkvo[4];
  ga::Workspace w;
  block_ws_layout(s, N, workspace, qkvo, &w);
  hipStream_t st = (hipStream_t)stream;
  GA_LAUNCH(ga::launch_project(0, s.B, s.n, s.H, X, Wqkv, qkvo[0], qkvo[1], qkvo[2], st), "projection launch");
  GA_TRY(run_forward(dims_of(s, N), qkvo[0], qkvo[1], qkvo[2], iters, scale, qkvo[3], nullptr, nullptr, nullptr, w,
                     st));
  GA_LAUNCH(ga::launch_project(1, s.B, s.n, s.H, qkvo[3], Wo, Y, nullptr, nullptr, st), "projection launch");
  return GA_OK;
}

int ga_merge_plan(ga_shape_t s, const void* Q, const void* K, const int32_t* belong, const float* centroid,
                  const int32_t* count, int32_t N, float scale, double eps, double* radius, double* dthr,
                  int32_t* partner, int32_t* merges, void* stream) {
  bool empty;
  GA_TRY(check_shape(s, N, &empty));
  if (!isfinite(scale)) return fail(GA_ERR_INVALID_ARG, "scale must be finite");
  if (!(eps > 1.0) || !isfinite(eps)) return fail(GA_ERR_INVALID_ARG, "eps must be a finite bound > 1 (got %g)", eps);
  if (N > ga::merge_max_groups())
    return fail(GA_ERR_UNSUPPORTED, "the merge plan supports N <= %d (got %d)", ga::merge_max_groups(), N);
  GA_TRY(check_ptr(Q, "Q", true));
  GA_TRY(check_ptr(K, "K", true));
  GA_TRY(check_ptr(belong, "belong", true));
  GA_TRY(check_ptr(centroid, "centroid", true));
  GA_TRY(check_ptr(count, "count", true));
  GA_TRY(check_ptr(radius, "radius", true));
  GA_TRY(check_ptr(dthr, "dthr", true));
  GA_TRY(check_ptr(partner, "partner", true));
  GA_TRY(check_ptr(merges, "merges", true));
  if (empty) return GA_OK;
  GA_LAUNCH(ga::launch_merge_plan(dims_of(s, N), Q, K, belong, centroid, count, fabs((double)scale), log(eps), radius,
                                  dthr, partner, merges, (hipStream_t)stream),
            "merge-plan launch");
  return GA_OK;
}

int32_t ga_next_group_count(int32_t N, const int32_t* merges, int64_t slices, double alpha) {
  if (N < 1) return fail(GA_ERR_INVALID_ARG, "N must be >= 1 (got %d)", N), 0;
  if (!(alpha >= 0.0 && alpha <= 1.0)) return fail(GA_ERR_INVALID_ARG, "alpha must lie in [0, 1]"), 0;
  if (slices < 0 || (slices > 0 && !merges)) return fail(GA_ERR_INVALID_ARG, "merges must hold `slices` counts"), 0;
  int64_t D = 0;
  for (int64_t u = 0; u < slices; ++u) D = u == 0 || merges[u] < D ? merges[u] : D;
  const double x = alpha * (double)(N - D) + (1.0 - alpha) * (double)N;
  const double r = floor(x + 0.5);
  return r < 1.0 ? 1 : (r > N ? N : (int32_t)r);
}

size_t ga_backward_workspace_bytes(ga_shape_t s, int32_t N) {
  bool empty;
  const std::string keep = g_last_error;
  const int rc = check_shape(s, N, &empty);
  g_last_error = keep;
  if (rc != GA_OK || s.dtype != GA_BF16 || N > ga::backward_max_groups()) return 0;
  return ga::backward_workspace_layout(dims_of(s, N), nullptr, nullptr);
}

int ga_backward(ga_shape_t s, const void* Q, const void* dO, const int32_t* belong, const float* centroid,
                const int32_t* count, const float* vsum, int32_t N, float scale, void* dQ, void* dK, void* dV,
                void* workspace, size_t workspace_bytes, void* stream) {
  bool empty;
  GA_TRY(check_shape(s, N, &empty));
  if (s.dtype != GA_BF16) return fail(GA_ERR_UNSUPPORTED, "the backward pass is bf16 only");
  if (N > ga::backward_max_groups())
    return fail(GA_ERR_UNSUPPORTED, "the backward pass supports N <= %d (got %d)", ga::backward_max_groups(), N);
  if (!isfinite(scale)) return fail(GA_ERR_INVALID_ARG, "scale must be finite");
  GA_TRY(check_ptr(Q, "Q", true));
  GA_TRY(check_ptr(dO, "dO", true));
  GA_TRY(check_ptr(belong, "belong", true));
  GA_TRY(check_ptr(centroid, "centroid", true));
  GA_TRY(check_ptr(count, "count", true));
  GA_TRY(check_ptr(vsum, "vsum", true));
  GA_TRY(check_ptr(dQ, "dQ", true));
  GA_TRY(check_ptr(dK, "dK", true));
  GA_TRY(check_ptr(dV, "dV", true));
  if (empty) return GA_OK;
  const ga::Dims d = dims_of(s, N);
  const size_t need = ga::backward_workspace_layout(d, nullptr, nullptr);
  if (!workspace) return fail(GA_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (((uintptr_t)workspace & 255u) != 0) return fail(GA_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  if (workspace_bytes < need)
    return fail(GA_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", workspace_bytes, need);
  ga::BackwardWorkspace w;
  ga::backward_workspace_layout(d, &w, workspace);
  GA_LAUNCH(ga::launch_backward(d, Q, dO, belong, centroid, count, vsum, scale, dQ, dK, dV, w, (hipStream_t)stream),
            "backward launch");
  return GA_OK;
}

const char* ga_status_string(int status) {
  switch (status) {
    case GA_OK: return "GA_OK";
    case GA_ERR_INVALID_ARG: return "GA_ERR_INVALID_ARG";
    case GA_ERR_UNSUPPORTED: return "GA_ERR_UNSUPPORTED";
    case GA_ERR_WORKSPACE: return "GA_ERR_WORKSPACE";
    case GA_ERR_HIP: return "GA_ERR_HIP";
    default: return "GA_ERR_UNKNOWN";
  }
}

const char* ga_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
