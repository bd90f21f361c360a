// C ABI of the depth-sparse layer library: argument checks, workspace plan,
// the launch sequence of one sparse layer and of the stack, the host-side
// retention allocation (Eqs. 5-8), and per-launch event timing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "adadsf.h"
#include "dsf_internal.h"

using namespace dsf;

// ------------------------------------------------------------------ errors

static thread_local std::string g_err;

static int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define DSF_CHECK(cond, code, ...) \
  do {                             \
    if (!(cond)) return fail(code, __VA_ARGS__); \
  } while (0)

#define DSF_HIP(expr)                                                              \
  do {                                                                             \
    hipError_t e_ = (expr);                                                        \
    if (e_ != hipSuccess) return fail(DSF_EHIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

extern "C" int dsf_version(void) { return DSF_VERSION; }
extern "C" const char* dsf_last_error(void) { return g_err.c_str(); }

static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// The current device must exist and be gfx950 (the only code object built).
static int check_device() {
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || n <= 0) {
    (void)hipGetLastError();
    return fail(DSF_ENODEVICE, "no GPU is visible");
  }
  int dev = 0;
  DSF_HIP(hipGetDevice(&dev));
  static std::mutex mu;
  static std::vector<int> arch_ok;  // -1 unknown, 0 no, 1 yes
  std::lock_guard<std::mutex> lock(mu);
  if (int(arch_ok.size()) < n) arch_ok.resize(n, -1);
  if (arch_ok[dev] < 0) {
    hipDeviceProp_t prop;
    DSF_HIP(hipGetDeviceProperties(&prop, dev));
    arch_ok[dev] = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 0;
  }
  if (!arch_ok[dev]) return fail(DSF_EUNSUPPORTED, "device %d is not gfx950 (MI355X)", dev);
  return DSF_OK;
}

static int check_dtype(int dtype) {
  DSF_CHECK(dtype == DSF_F32 || dtype == DSF_BF16, DSF_EUNSUPPORTED, "dtype %d is not DSF_F32 or DSF_BF16", dtype);
  return DSF_OK;
}

static size_t elem_bytes(int dtype) { return dtype == DSF_BF16 ? 2 : 4; }

// --------------------------------------------------------------- timing

namespace {
struct TimingRec {
  int kind;
  hipEvent_t start, stop;
  bool deferred;  // opened without a start event: the launcher records both (timing_claim)
  bool claimed;
};
std::mutex g_tmu;
std::vector<TimingRec> g_recs;
size_t g_used = 0;
long g_open = -1;
uint32_t g_mask = 0;
}  // namespace

namespace dsf {
void timing_begin(int kind, hipStream_t s, bool deferred) {
  std::lock_guard<std::mutex> lock(g_tmu);
  if (g_used >= g_recs.size() || g_open >= 0 || !((g_mask >> kind) & 1u)) return;
  TimingRec& r = g_recs[g_used];
  r.kind = kind;
  r.deferred = deferred;
  r.claimed = false;
  if (deferred || hipEventRecord(r.start, s) == hipSuccess) g_open = long(g_used);
}
bool timing_claim(hipEvent_t* start, hipEvent_t* stop) {
  std::lock_guard<std::mutex> lock(g_tmu);
  if (g_open < 0) return false;
  TimingRec& r = g_recs[g_open];
  if (!r.deferred || r.claimed) return false;
  r.claimed = true;
  *start = r.start;
  *stop = r.stop;
  return true;
}
void timing_continue() {
  std::lock_guard<std::mutex> lock(g_tmu);
  if (g_open < 0) return;
  TimingRec& r = g_recs[g_open];
  if (!r.deferred || !r.claimed) return;
  const int kind = r.kind;
  ++g_used;
  g_open = -1;
  if (g_used >= g_recs.size()) return;
  TimingRec& n = g_recs[g_used];
  n.kind = kind;
  n.deferred = true;
  n.claimed = false;
  g_open = long(g_used);
}
void timing_end(int kind, hipStream_t s) {
  std::lock_guard<std::mutex> lock(g_tmu);
  if (g_open < 0 || g_recs[g_open].kind != kind) return;
  TimingRec& r = g_recs[g_open];
  if (r.deferred ? r.claimed : hipEventRecord(r.stop, s) == hipSuccess) ++g_used;
  g_open = -1;
}
}  // namespace dsf

extern "C" int dsf_timing_enable(int max_records, uint32_t kind_mask) {
  DSF_CHECK(max_records >= 0, DSF_EINVAL, "max_records < 0");
  std::lock_guard<std::mutex> lock(g_tmu);
  for (auto& r : g_recs) {
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  g_recs.clear();
  g_used = 0;
  g_open = -1;
  g_mask = kind_mask;
  if (max_records == 0) return DSF_OK;
  int rc = check_device();
  if (rc) return rc;
  g_recs.resize(size_t(max_records));
  for (auto& r : g_recs) {
    r.kind = -1;
    r.deferred = r.claimed = false;
    DSF_HIP(hipEventCreate(&r.start));
    DSF_HIP(hipEventCreate(&r.stop));
  }
  return DSF_OK;
}

extern "C" int dsf_timing_read(int kind, int* launches, double* total_ms) {
  DSF_CHECK(launches && total_ms, DSF_EINVAL, "null output pointer");
  DSF_CHECK(kind >= 0 && kind < DSF_KIND_COUNT, DSF_EINVAL, "unknown kernel kind %d", kind);
  std::lock_guard<std::mutex> lock(g_tmu);
  int cnt = 0;
  double tot = 0.0;
  for (size_t i = 0; i < g_used; ++i) {
    if (g_recs[i].kind != kind) continue;
    DSF_HIP(hipEventSynchronize(g_recs[i].stop));
    float ms = 0.f;
    DSF_HIP(hipEventElapsedTime(&ms, g_recs[i].start, g_recs[i].stop));
    tot += ms;
    ++cnt;
    g_recs[i].kind = -1;
  }
  *launches = cnt;
  *total_ms = tot;
  return DSF_OK;
}

// ---------------------------------------------- retention allocation, host

extern "C" int dsf_retention_from_similarity(const double* s, int L, double t, double tau, double beta,
                                             int clip_mode, double* r_out) {
  DSF_CHECK(s && r_out, DSF_EINVAL, "null pointer");
  DSF_CHECK(L >= 1, DSF_EINVAL, "L must be >= 1");
  DSF_CHECK(t > 0.0 && t <= 1.0, DSF_EINVAL, "target retention t must be in (0, 1]");
  DSF_CHECK(beta > 0.0 && std::isfinite(beta), DSF_EINVAL, "beta must be positive");
  DSF_CHECK(clip_mode >= DSF_CLIP_NONE && clip_mode <= DSF_CLIP_BUDGET, DSF_EINVAL, "unknown clip mode");
  for (int i = 0; i < L; ++i) DSF_CHECK(std::isfinite(s[i]), DSF_EINVAL, "s[%d] is not finite", i);
  if (!(tau > 0.0)) {  // no temperature: uniform allocation
    for (int i = 0; i < L; ++i) r_out[i] = t;
    return DSF_OK;
  }
  std::vector<double> w(L), rp(L), r(L);
  double smax = s[0];
  for (int i = 1; i < L; ++i) smax = s[i] > smax ? s[i] : smax;
  double wsum = 0.0;
  for (int i = 0; i < L; ++i) {  // Eq. 5
    w[i] = std::exp((s[i] - smax) / tau);
    wsum += w[i];
  }
  double wmean = 0.0;
  for (int i = 0; i < L; ++i) {
    w[i] /= wsum;
    wmean += w[i];
  }
  wmean /= L;
  double rpsum = 0.0;
  for (int i = 0; i < L; ++i) {
    const double z = beta * (wmean - w[i]);        // Eq. 6
    rp[i] = 0.05 + 0.9 / (1.0 + std::exp(-z));     // Eq. 7
    rpsum += rp[i];
  }
  for (int i = 0; i < L; ++i) r[i] = t * L / rpsum * rp[i];  // Eq. 8
  if (clip_mode == DSF_CLIP_PLAIN) {
    for (int i = 0; i < L; ++i) r[i] = r[i] > 1.0 ? 1.0 : r[i];
  } else if (clip_mode == DSF_CLIP_BUDGET) {
    std::vector<char> capped(L, 0);
    for (;;) {
      bool over = false;
      for (int i = 0; i < L; ++i)
        if (r[i] > 1.0) {
          capped[i] = 1;
          over = true;
        }
      if (!over) break;
      int ncap = 0;
      double free_rp = 0.0;
      for (int i = 0; i < L; ++i) {
        if (capped[i]) ++ncap;
        else free_rp += rp[i];
      }
      const double budget = t * L - ncap;
      for (int i = 0; i < L; ++i) r[i] = capped[i] ? 1.0 : budget * rp[i] / free_rp;
    }
  }
  for (int i = 0; i < L; ++i) r_out[i] = r[i];
  return DSF_OK;
}

extern "C" int dsf_k_from_retention(double r, int T, int rounding) {
  if (!std::isfinite(r) || T < 0 || (rounding != DSF_ROUND_FLOOR && rounding != DSF_ROUND_CEIL)) {
    fail(DSF_EINVAL, "bad argument to dsf_k_from_retention");
    return -1;
  }
  const double x = r * double(T);
  double k = rounding == DSF_ROUND_FLOOR ? std::floor(x + 1e-6) : std::ceil(x - 1e-6);
  if (k < 0) k = 0;
  if (k > T) k = T;
  return int(k);
}

// ------------------------------------------------------ similarity, Eq. 4

extern "C" size_t dsf_sim_workspace_size(int64_t n_tokens) {
  if (n_tokens < 0) return 0;
  return ((size_t(sim_grid(n_tokens)) * sizeof(double) + 255) / 256) * 256;
}

extern "C" int dsf_sim_stats(const void* x_in, const void* x_out, int dtype, int64_t n_tokens, int d,
                             float* per_token_cos, double* accum, void* workspace, size_t workspace_bytes,
                             hipStream_t stream) {
  int rc = check_dtype(dtype);
  if (rc) return rc;
  DSF_CHECK(n_tokens >= 0, DSF_EINVAL, "n_tokens < 0");
  DSF_CHECK(d > 0 && d % 8 == 0, DSF_EUNSUPPORTED, "d must be a positive multiple of 8");
  if (n_tokens == 0) return DSF_OK;
  DSF_CHECK(x_in && x_out && accum, DSF_EINVAL, "null pointer");
  DSF_CHECK(aligned16(x_in) && aligned16(x_out), DSF_EINVAL, "x_in / x_out must be 16-byte aligned");
  DSF_CHECK(workspace && workspace_bytes >= dsf_sim_workspace_size(n_tokens), DSF_EWORKSPACE,
            "workspace needs %zu bytes", dsf_sim_workspace_size(n_tokens));
  rc = check_device();
  if (rc) return rc;
  DSF_HIP(launch_sim_stats(dtype, x_in, x_out, n_tokens, d, per_token_cos, (double*)workspace, accum, stream));
  return DSF_OK;
}

extern "C" int dsf_sim_finalize(const double* accum_dev, int L, double* s_host, hipStream_t stream) {
  DSF_CHECK(L >= 0, DSF_EINVAL, "L < 0");
  if (L == 0) return DSF_OK;
  DSF_CHECK(accum_dev && s_host, DSF_EINVAL, "null pointer");
  int rc = check_device();
  if (rc) return rc;
  std::vector<double> buf(size_t(L) * 2);
  DSF_HIP(hipMemcpyAsync(buf.data(), accum_dev, buf.size() * sizeof(double), hipMemcpyDeviceToHost, stream));
  DSF_HIP(hipStreamSynchronize(stream));
  for (int l = 0; l < L; ++l) s_host[l] = buf[2 * l] / buf[2 * l + 1];
  return DSF_OK;
}

// ------------------------------------------------------------ routing

extern "C" int dsf_router_score(const void* x, int dtype, int64_t n_tokens, int d, int d_r, const void* w1,
                                const void* b1, const void* w2, float b2, float* scores, hipStream_t stream) {
  int rc = check_dtype(dtype);
  if (rc) return rc;
  DSF_CHECK(n_tokens >= 0 && n_tokens < (int64_t(1) << 40), DSF_EINVAL, "bad n_tokens");
  DSF_CHECK(d > 0 && d % 8 == 0, DSF_EUNSUPPORTED, "d must be a positive multiple of 8");
  DSF_CHECK(d_r == 16 || d_r == 32 || d_r == 48 || d_r == 64, DSF_EUNSUPPORTED, "d_r must be 16, 32, 48 or 64");
  if (n_tokens == 0) return DSF_OK;
  DSF_CHECK(x && w1 && w2 && scores, DSF_EINVAL, "null pointer");
  DSF_CHECK(aligned16(x) && aligned16(w1), DSF_EINVAL, "x and W1 must be 16-byte aligned");
  rc = check_device();
  if (rc) return rc;
  DSF_HIP(launch_router(dtype, x, n_tokens, d, d_r, w1, b1, w2, b2, scores, stream));
  return DSF_OK;
}

// ------------------------------------------- router-score pathway (training)

extern "C" int dsf_gate_score_grad(const void* dy, const void* x_in, const void* x_out, int dtype,
                                   const float* scores, const int32_t* idx, int B, int T, int k, int d,
                                   float* dscore, hipStream_t stream) {
  int rc = check_dtype(dtype);
  if (rc) return rc;
  DSF_CHECK(B >= 0 && T >= 0, DSF_EINVAL, "B and T must be >= 0");
  DSF_CHECK(int64_t(B) * T < (int64_t(1) << 31), DSF_EINVAL, "B * T too large");
  DSF_CHECK(k >= 0 && k <= T, DSF_EINVAL, "k=%d outside [0, T=%d]", k, T);
  DSF_CHECK(d > 0 && d % 8 == 0, DSF_EUNSUPPORTED, "d must be a positive multiple of 8");
  if (B == 0 || T == 0) return DSF_OK;
  DSF_CHECK(dscore, DSF_EINVAL, "dscore is null");
  if (k > 0) {
    DSF_CHECK(dy && x_in && x_out && scores && idx, DSF_EINVAL, "null pointer");
    DSF_CHECK(aligned16(dy) && aligned16(x_in) && aligned16(x_out), DSF_EINVAL,
              "dy, x_in and x_out must be 16-byte aligned");
  }
  rc = check_device();
  if (rc) return rc;
  DSF_HIP(launch_gate_grad(dtype, dy, x_in, x_out, scores, idx, B, T, k, d, dscore, stream));
  return DSF_OK;
}

static bool router_width_ok(int d_r) { return d_r == 16 || d_r == 32 || d_r == 48 || d_r == 64; }

extern "C" size_t dsf_router_backward_workspace_size(int64_t n_tokens, int d, int d_r) {
  if (n_tokens < 0 || n_tokens >= (int64_t(1) << 31) || d <= 0 || d % 8 != 0 || !router_width_ok(d_r)) return 0;
  return router_bwd_workspace_bytes(n_tokens, d, d_r);
}

extern "C" int dsf_router_backward(const void* x, int dtype, int64_t n_tokens, int d, int d_r, const void* w1,
                                   const void* b1, const void* w2, const float* dscore, float* dw1, float* db1,
                                   float* dw2, float* db2, void* dx, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream) {
  int rc = check_dtype(dtype);
  if (rc) return rc;
  DSF_CHECK(n_tokens >= 0 && n_tokens < (int64_t(1) << 31), DSF_EINVAL, "bad n_tokens");
  DSF_CHECK(d > 0 && d % 8 == 0, DSF_EUNSUPPORTED, "d must be a positive multiple of 8");
  DSF_CHECK(router_width_ok(d_r), DSF_EUNSUPPORTED, "d_r must be 16, 32, 48 or 64");
  DSF_CHECK(w1 && w2 && dw1 && dw2 && db2, DSF_EINVAL, "null pointer");
  DSF_CHECK(!db1 || b1, DSF_EINVAL, "db1 needs b1");
  if (n_tokens > 0) {
    DSF_CHECK(x && dscore, DSF_EINVAL, "null pointer");
    DSF_CHECK(aligned16(x) && aligned16(w1) && (!dx || aligned16(dx)), DSF_EINVAL,
              "x, W1 and dx must be 16-byte aligned");
    const size_t need = router_bwd_workspace_bytes(n_tokens, d, d_r);
    DSF_CHECK(workspace_bytes >= need, DSF_EWORKSPACE, "workspace needs %zu bytes, got %zu", need,
              workspace_bytes);
    DSF_CHECK(workspace && (reinterpret_cast<uintptr_t>(workspace) & 255u) == 0, DSF_EINVAL,
              "workspace must be non-null and 256-byte aligned");
  }
  rc = check_device();
  if (rc) return rc;
  if (n_tokens == 0) {  // empty sums: every gradient is zero
    DSF_HIP(launch_zero_u32(reinterpret_cast<uint32_t*>(dw1), int64_t(d_r) * d, stream));
    if (db1) DSF_HIP(launch_zero_u32(reinterpret_cast<uint32_t*>(db1), d_r, stream));
    DSF_HIP(launch_zero_u32(reinterpret_cast<uint32_t*>(dw2), d_r, stream));
    DSF_HIP(launch_zero_u32(reinterpret_cast<uint32_t*>(db2), 1, stream));
    return DSF_OK;
  }
  RouterBwdArgs a{};
  a.dtype = dtype;
  a.x = x; a.n = n_tokens; a.d = d; a.d_r = d_r;
  a.w1 = w1; a.b1 = b1; a.w2 = w2;
  a.dscore = dscore;
  a.dw1 = dw1; a.db1 = db1; a.dw2 = dw2; a.db2 = db2;
  a.dx = dx;
  a.workspace = workspace;
  DSF_HIP(launch_router_backward(a, stream));
  return DSF_OK;
}

extern "C" int dsf_topk_select(const float* scores, int B, int T, int k, int32_t* idx, hipStream_t stream) {
  DSF_CHECK(B >= 0 && T >= 0, DSF_EINVAL, "B and T must be >= 0");
  DSF_CHECK(k >= 0 && k <= T, DSF_EINVAL, "k=%d outside [0, T=%d]", k, T);
  if (B == 0 || k == 0) return DSF_OK;
  DSF_CHECK(scores && idx, DSF_EINVAL, "null pointer");
  int rc = check_device();
  if (rc) return rc;
  DSF_HIP(launch_topk(scores, B, T, k, idx, stream));
  return DSF_OK;
}

static int check_rows(const void* x, const void* other, int dtype, int B, int T, int d, const int32_t* idx, int k) {
  int rc = check_dtype(dtype);
  if (rc) return rc;
  DSF_CHECK(B >= 0 && T >= 0, DSF_EINVAL, "B and T must be >= 0");
  DSF_CHECK(int64_t(B) * T < (int64_t(1) << 31), DSF_EINVAL, "B * T too large");
  DSF_CHECK(k >= 0 && k <= T, DSF_EINVAL, "k=%d outside [0, T=%d]", k, T);
  DSF_CHECK(d > 0 && d % 8 == 0, DSF_EUNSUPPORTED, "d must be a positive multiple of 8");
  if (B == 0 || k == 0) return DSF_OK;
  DSF_CHECK(x && other && idx, DSF_EINVAL, "null pointer");
  DSF_CHECK(aligned16(x) && aligned16(other), DSF_EINVAL, "row buffers must be 16-byte aligned");
  return DSF_OK;
}

extern "C" int dsf_gather_rows(const void* x, int dtype, int B, int T, int d, const int32_t* idx, int k, void* out,
                               hipStream_t stream) {
  int rc = check_rows(x, out, dtype, B, T, d, idx, k);
  if (rc || B == 0 || k == 0) return rc;
  rc = check_device();
  if (rc) return rc;
  DSF_HIP(launch_gather(dtype, x, B, T, d, idx, k, out, stream));
  return DSF_OK;
}

extern "C" int dsf_scatter_residual(void* x, const void* delta, int dtype, int B, int T, int d, const int32_t* idx,
                                    int k, hipStream_t stream) {
  int rc = check_rows(x, delta, dtype, B, T, d, idx, k);
  if (rc || B == 0 || k == 0) return rc;
  rc = check_device();
  if (rc) return rc;
  DSF_HIP(launch_scatter(dtype, x, delta, B, T, d, idx, k, stream));
  return DSF_OK;
}

extern "C" int dsf_attention_forward(const void* q, const void* k, const void* v, int dtype, int B, int Hq,
                                     int Hkv, int n, int hd, void* out, hipStream_t stream) {
  int rc = check_dtype(dtype);
  if (rc) return rc;
  DSF_CHECK(B >= 0 && n >= 0, DSF_EINVAL, "B and n must be >= 0");
  DSF_CHECK(Hq > 0 && Hkv > 0 && Hq % Hkv == 0, DSF_EINVAL, "need Hq %% Hkv == 0");
  DSF_CHECK(hd == 32 || hd == 64 || hd == 128, DSF_EUNSUPPORTED, "head_dim must be 32, 64 or 128");
  DSF_CHECK(int64_t(B) * n * Hq < (int64_t(1) << 31), DSF_EINVAL, "problem too large");
  if (B == 0 || n == 0) return DSF_OK;
  DSF_CHECK(q && k && v && out, DSF_EINVAL, "null pointer");
  DSF_CHECK(aligned16(q) && aligned16(k) && aligned16(v) && aligned16(out), DSF_EINVAL,
            "q, k, v and out must be 16-byte aligned");
  rc = check_device();
  if (rc) return rc;
  DSF_HIP(launch_attention(dtype, q, k, v, B, Hq, Hkv, n, hd, out, stream));
  return DSF_OK;
}

// ------------------------------------------------------- workspace plan

namespace {
struct Plan {
  size_t ctl, scores, idx, a1, a2, q, k, v, attn, act, h, m2, rope, xin, simpart, alignpart, skpart, total;
};

// Control block at offset 0 of a layer/stack workspace, zeroed by one launch
// at the start of every call: word 0 is the call's status word (read by
// dsf_workspace_status), then the stream-K flags, then the per-sequence
// counters of the router + Top-K launch.
constexpr int kCtlFlagsWord = 64;
size_t ctl_words(int B) { return size_t(kCtlFlagsWord) + size_t(gemm_flag_count()) + size_t(B); }

size_t up256(size_t x) { return (x + 255) / 256 * 256; }

Plan make_plan(const dsf_layer_desc& D, int dtype, int B, int T, int k_max, bool with_sim,
               bool with_align = false) {
  const size_t eb = elem_bytes(dtype);
  const size_t N = size_t(B) * size_t(k_max);
  const bool qwen = D.block == DSF_BLOCK_QWEN_SEQ;
  Plan p{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += up256(bytes);
    return o;
  };
  p.ctl = take(sizeof(uint32_t) * ctl_words(B));
  p.scores = take(4 * size_t(B) * T);
  p.idx = take(4 * N);
  p.a1 = take(eb * N * D.d_model);
  p.a2 = qwen ? 0 : take(eb * N * D.d_model);
  p.q = take(eb * N * D.n_heads * D.head_dim);
  p.k = take(eb * N * D.n_kv_heads * D.head_dim);
  p.v = take(eb * N * D.n_kv_heads * D.head_dim);
  p.attn = take(eb * N * D.n_heads * D.head_dim);
  p.act = take(eb * N * D.d_ff);
  p.h = qwen ? take(eb * N * D.d_model) : 0;
  p.m2 = qwen ? take(eb * N * D.d_model) : 0;
  p.rope = take(4 * size_t(T) * D.rotary_dims);
  p.xin = with_sim ? take(eb * size_t(B) * T * D.d_model) : 0;
  p.simpart = with_sim ? take(dsf_sim_workspace_size(int64_t(B) * T)) : 0;
  p.alignpart = with_align ? take(sizeof(double) * size_t(align_grid(int64_t(B) * T))) : 0;
  // stream-K partial tiles (bf16 GEMMs); their flags are in the control block
  p.skpart = dtype == DSF_BF16 ? take(gemm_partial_bytes()) : 0;
  p.total = off;
  return p;
}

int check_desc(const dsf_layer_desc* D) {
  DSF_CHECK(D, DSF_EINVAL, "null layer descriptor");
  DSF_CHECK(D->block == DSF_BLOCK_NEOX_PARALLEL || D->block == DSF_BLOCK_QWEN_SEQ, DSF_EUNSUPPORTED,
            "unknown block template %d", D->block);
  DSF_CHECK(D->d_model > 0 && D->d_model % 8 == 0, DSF_EUNSUPPORTED, "d_model must be a positive multiple of 8");
  DSF_CHECK(D->d_model <= 8192, DSF_EUNSUPPORTED, "d_model above 8192");
  DSF_CHECK(D->n_heads > 0 && D->n_kv_heads > 0 && D->n_heads % D->n_kv_heads == 0, DSF_EINVAL,
            "need n_heads %% n_kv_heads == 0");
  DSF_CHECK(D->head_dim == 32 || D->head_dim == 64 || D->head_dim == 128, DSF_EUNSUPPORTED,
            "head_dim must be 32, 64 or 128");
  DSF_CHECK(D->d_ff > 0 && D->d_ff % 64 == 0, DSF_EUNSUPPORTED, "d_ff must be a positive multiple of 64");
  DSF_CHECK(D->rotary_dims > 0 && D->rotary_dims % 2 == 0 && D->rotary_dims <= D->head_dim, DSF_EINVAL,
            "rotary_dims must be even and in (0, head_dim]");
  DSF_CHECK(D->d_router == 16 || D->d_router == 32 || D->d_router == 48 || D->d_router == 64, DSF_EUNSUPPORTED,
            "d_router must be 16, 32, 48 or 64");
  DSF_CHECK(D->norm_eps > 0.f && std::isfinite(D->norm_eps), DSF_EINVAL, "norm_eps must be positive");
  DSF_CHECK(D->rope_theta > 0.0 && std::isfinite(D->rope_theta), DSF_EINVAL, "rope_theta must be positive");
  DSF_CHECK(D->reserved == 0.f, DSF_EINVAL, "reserved field must be 0");
  return DSF_OK;
}

int check_weights(const dsf_layer_desc& D, const dsf_layer_weights* W, int l) {
  DSF_CHECK(W, DSF_EINVAL, "null weights (layer %d)", l);
  const void* req[] = {W->router_w1, W->router_w2, W->norm1_w, W->norm2_w, W->w_qkv, W->w_o, W->w_up, W->w_down};
  const char* nm[] = {"router_w1", "router_w2", "norm1_w", "norm2_w", "w_qkv", "w_o", "w_up", "w_down"};
  for (int i = 0; i < 8; ++i) {
    DSF_CHECK(req[i], DSF_EINVAL, "layer %d: %s is null", l, nm[i]);
    DSF_CHECK(aligned16(req[i]), DSF_EINVAL, "layer %d: %s is not 16-byte aligned", l, nm[i]);
  }
  const void* opt[] = {W->router_b1, W->norm1_b, W->norm2_b, W->b_qkv, W->b_o, W->b_up, W->b_down};
  for (const void* p : opt) DSF_CHECK(aligned16(p), DSF_EINVAL, "layer %d: a bias is not 16-byte aligned", l);
  if (D.block == DSF_BLOCK_QWEN_SEQ)
    DSF_CHECK(!W->norm1_b && !W->norm2_b, DSF_EINVAL, "layer %d: RMSNorm takes no bias", l);
  DSF_CHECK(W->reserved == 0.f, DSF_EINVAL, "layer %d: reserved field must be 0", l);
  return DSF_OK;
}
}  // namespace

extern "C" size_t dsf_workspace_size(const dsf_layer_desc* desc, int dtype, int B, int T, int k_max,
                                     int with_similarity) {
  if (check_desc(desc) || check_dtype(dtype) || B < 0 || T < 0 || k_max < 0 || k_max > T) return 0;
  return make_plan(*desc, dtype, B, T, k_max, with_similarity != 0).total;
}

extern "C" int dsf_workspace_status(const void* workspace, uint32_t* status, hipStream_t stream) {
  DSF_CHECK(workspace && status, DSF_EINVAL, "null workspace or status pointer");
  uint32_t v = 0;
  DSF_HIP(hipMemcpyAsync(&v, workspace, sizeof(v), hipMemcpyDeviceToHost, stream));
  DSF_HIP(hipStreamSynchronize(stream));
  *status = v;
  return DSF_OK;
}

// --------------------------------------------------- one sparse layer

namespace {
// A second stream for work that the block's data flow lets run beside the
// main chain: the NeoX FFN up projection needs only LN2 of the kept rows, so
// it runs while QKV and attention run on the caller's stream. One per device
// and host thread, created on the thread's first such call, non-blocking,
// default priority, and destroyed with its events when the thread exits (a
// per-thread stream never joins another thread's graph capture). Fork and
// join are event waits, which a caller capturing the stream into a graph
// records as well. DSF_SINGLE_STREAM=1 (read at every call) keeps everything
// on one stream.
// The fork and join events only order the two streams of one device: the
// kernels' own end-of-kernel releases make their results visible device-wide,
// so the events skip the system-scope fence (measured 1.2 % per stack step).
constexpr unsigned kAuxEventFlags = hipEventDisableTiming | hipEventDisableSystemFence;
struct AuxStream {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};

// The calling thread's streams, one slot per device. Thread-local objects
// of a thread are destroyed when it exits, before the HIP runtime's own
// teardown at process exit; a stream with work still queued is released once
// that work completes. Errors at that point have no caller to go to.
struct AuxStreams {
  std::vector<AuxStream> per_dev;
  ~AuxStreams() {
    for (AuxStream& a : per_dev) {
      if (a.fork) (void)hipEventDestroy(a.fork);
      if (a.join) (void)hipEventDestroy(a.join);
      if (a.s) (void)hipStreamDestroy(a.s);
    }
  }
};

int get_aux(const AuxStream** out) {
  *out = nullptr;
  const char* e = getenv("DSF_SINGLE_STREAM");
  if (e && e[0] == '1') return DSF_OK;
  static thread_local AuxStreams streams;
  std::vector<AuxStream>& per_dev = streams.per_dev;
  int dev = 0;
  DSF_HIP(hipGetDevice(&dev));
  if (dev < 0) return fail(DSF_EHIP, "bad device %d", dev);
  if (size_t(dev) >= per_dev.size()) per_dev.resize(size_t(dev) + 1);
  AuxStream& a = per_dev[size_t(dev)];
  if (!a.s || !a.fork || !a.join) {  // created together; a partial set is retried whole
    AuxStream n;
    hipError_t err = hipStreamCreateWithFlags(&n.s, hipStreamNonBlocking);
    if (err == hipSuccess) err = hipEventCreateWithFlags(&n.fork, kAuxEventFlags);
    if (err == hipSuccess) err = hipEventCreateWithFlags(&n.join, kAuxEventFlags);
    if (err != hipSuccess) {
      if (n.fork) (void)hipEventDestroy(n.fork);
      if (n.s) (void)hipStreamDestroy(n.s);
      return fail(DSF_EHIP, "creating the second stream: %s", hipGetErrorString(err));
    }
    a = n;
  }
  *out = &a;
  return DSF_OK;
}

struct Ctx {
  const dsf_layer_desc* D;
  int dtype, B, T;
  char* ws;
  Plan plan;
  hipStream_t s;
  mutable uint32_t epoch;  // last stream-K epoch handed out since the flags were zeroed
  const AuxStream* aux;    // null: one stream
};

uint32_t* at_status(const Ctx& c) { return reinterpret_cast<uint32_t*>(c.ws + c.plan.ctl); }
uint32_t* at_flags(const Ctx& c) { return at_status(c) + kCtlFlagsWord; }
// per-sequence counters of the router + Top-K launch (bf16), after the flags
uint32_t* at_route_count(const Ctx& c) { return at_flags(c) + gemm_flag_count(); }

// Zero the control block at the start of a call (one launch): the status
// word, the stream-K flags and the router counters. GEMM launches then take
// epochs 1, 2, ... (the flags of a finished launch never equal a later
// epoch), and each router + Top-K launch leaves its counters zero again.
int reset_stream_k(const Ctx& c) {
  c.epoch = 0;
  DSF_HIP(launch_zero_u32(at_status(c), int64_t(ctl_words(c.B)), c.s));
  return DSF_OK;
}

// Router and Top-K in one launch up to this many tokens per sequence: there
// the saved launch pays; beyond it the Top-K of the last-arriving router
// workgroup (512 threads) is slower than the separate 1024-thread kernel
// (Qwen2.5-7B shape, T 8192: 3.09 against 2.27 + 0.46 ms per step).
// DSF_UNFUSED_ROUTING=1 (read at every call) always runs two launches.
constexpr int kFusedRoutingMaxT = 4096;
bool fused_routing(int T) {
  const char* e = getenv("DSF_UNFUSED_ROUTING");
  return !(e && e[0] == '1') && T <= kFusedRoutingMaxT;
}

// The stream-K fields of a GEMM launch on this call's workspace.
void use_stream_k(const Ctx& c, GemmArgs& g) {
  if (c.dtype != DSF_BF16) return;
  g.part = reinterpret_cast<float*>(c.ws + c.plan.skpart);
  g.flags = at_flags(c);
  g.status = at_status(c);
  g.epoch = ++c.epoch;
}

template <typename P>
P* at(const Ctx& c, size_t off) {
  return reinterpret_cast<P*>(c.ws + off);
}

// Enqueue one layer. k > 0. dense: every token at positions 0..T-1.
int run_layer(const Ctx& c, const dsf_layer_weights* W, void* x, int k, bool dense, bool gate, float* scores_out,
              int32_t* idx_out, const int32_t* idx_in) {
  const dsf_layer_desc& D = *c.D;
  const int B = c.B, T = c.T, d = D.d_model;
  const int hd = D.head_dim, Hq = D.n_heads, Hkv = D.n_kv_heads, f = D.d_ff;
  const bool qwen = D.block == DSF_BLOCK_QWEN_SEQ;
  const int32_t* idx = nullptr;
  float* scores = nullptr;
  if (!dense && !idx_in && router_topk_fusable(c.dtype, T, D.d_router) && fused_routing(T)) {
    // router and Top-K in one launch (its last workgroup of each sequence selects)
    scores = scores_out ? scores_out : at<float>(c, c.plan.scores);
    int32_t* dst = idx_out ? idx_out : at<int32_t>(c, c.plan.idx);
    DSF_HIP(launch_router_topk(x, B, T, d, D.d_router, W->router_w1, W->router_b1, W->router_w2, W->router_b2,
                               scores, k, dst, at_route_count(c), c.s));
    idx = dst;
  } else if (!dense) {
    scores = scores_out ? scores_out : at<float>(c, c.plan.scores);
    DSF_HIP(launch_router(c.dtype, x, int64_t(B) * T, d, D.d_router, W->router_w1, W->router_b1, W->router_w2,
                          W->router_b2, scores, c.s));
    if (idx_in) {
      idx = idx_in;
      if (idx_out) DSF_HIP(hipMemcpyAsync(idx_out, idx_in, sizeof(int32_t) * size_t(B) * k, hipMemcpyDeviceToDevice, c.s));
    } else {
      int32_t* dst = idx_out ? idx_out : at<int32_t>(c, c.plan.idx);
      DSF_HIP(launch_topk(scores, B, T, k, dst, c.s));
      idx = dst;
    }
  }
  const int kk = dense ? T : k;
  const int M = B * kk;
  const int dq = Hq * hd, dkv = Hkv * hd;

  NormArgs na{};
  na.dtype = c.dtype;
  na.src = x;
  na.src_rows = T;
  na.idx = idx;
  na.B = B;
  na.kk = kk;
  na.d = d;
  na.eps = D.norm_eps;
  na.rms = qwen;
  na.w1 = W->norm1_w;
  na.b1 = W->norm1_b;
  na.out1 = at<char>(c, c.plan.a1);
  if (!qwen) {
    na.w2 = W->norm2_w;
    na.b2 = W->norm2_b;
    na.out2 = at<char>(c, c.plan.a2);
  }
  DSF_HIP(launch_norm(na, c.s));

  GemmArgs g{};
  g.dtype = c.dtype;
  g.B = B;
  g.kk = kk;
  g.T = T;
  g.idx = idx;
  // NeoX: the FFN up projection reads only LN2 of the kept rows, so it runs
  // on the second stream beside QKV and attention, launched first so that
  // their workgroups fill the CU slots it leaves (never stream-K there: the
  // partial-sum workspace belongs to the main stream's GEMMs). Measured:
  // 3.59 against 3.64 ms per neox160m step; forking after QKV gained nothing.
  hipStream_t us = c.s;
  if (!qwen && c.aux) {
    DSF_HIP(hipEventRecord(c.aux->fork, c.s));
    DSF_HIP(hipStreamWaitEvent(c.aux->s, c.aux->fork, 0));
    us = c.aux->s;
  }
  // NeoX: the up and QKV projections share the chip; one tile size for both
  const int pair_hint = qwen ? 0 : gemm_pair_tile_hint(M, dq + 2 * dkv, d);
  if (!qwen) {  // FFN up + GELU on LN2 of the kept rows
    GemmArgs u = g;
    u.tile_hint = pair_hint;
    u.M = M; u.N = f; u.K = d; u.K1 = d;
    u.a = na.out2; u.lda = d;
    u.b = W->w_up; u.ldb = d;
    u.epi = EPI_BIAS_GELU; u.bias = W->b_up;
    u.out = at<char>(c, c.plan.act); u.ldo = f;
    TimedScope ts(DSF_KIND_GEMM_UP, us, true);
    if (us == c.s) use_stream_k(c, u);
    DSF_HIP(launch_gemm(u, us));
  }
  {  // QKV projection, bias, RoPE at the kept tokens' original positions
    GemmArgs q = g;
    q.M = M; q.N = dq + 2 * dkv; q.K = d; q.K1 = d;
    q.a = na.out1; q.lda = d;
    q.b = W->w_qkv; q.ldb = d;
    q.epi = EPI_QKV_ROPE;
    q.tile_hint = pair_hint;
    q.bias = W->b_qkv;
    q.q = at<char>(c, c.plan.q); q.k = at<char>(c, c.plan.k); q.v = at<char>(c, c.plan.v);
    q.Hq = Hq; q.Hkv = Hkv; q.hd = hd; q.R = D.rotary_dims;
    q.rope = at<float>(c, c.plan.rope);
    TimedScope ts(DSF_KIND_GEMM_QKV, c.s, true);
    use_stream_k(c, q);
    DSF_HIP(launch_gemm(q, c.s));
  }
  DSF_HIP(launch_attention(c.dtype, at<char>(c, c.plan.q), at<char>(c, c.plan.k), at<char>(c, c.plan.v), B, Hq,
                           Hkv, kk, hd, at<char>(c, c.plan.attn), c.s));
  if (!qwen) {
    if (us != c.s) {
      DSF_HIP(hipEventRecord(c.aux->join, us));
      DSF_HIP(hipStreamWaitEvent(c.s, c.aux->join, 0));
    }
    {  // parallel residual: [attn | act] . [W_o | W_down]^T + b_o + b_down + x, scattered back
      GemmArgs o = g;
      o.M = M; o.N = d; o.K = dq + f; o.K1 = dq;
      o.a = at<char>(c, c.plan.attn); o.lda = dq;
      o.a2 = at<char>(c, c.plan.act); o.lda2 = f;
      o.b = W->w_o; o.ldb = dq;
      o.b2 = W->w_down; o.ldb2 = f;
      o.epi = gate ? EPI_RESID_SCATTER_GATE : EPI_RESID_SCATTER; o.bias = W->b_o; o.bias2 = W->b_down;
      o.x = x; o.gate = scores;
      TimedScope ts(DSF_KIND_GEMM_DOWN, c.s, true);
      use_stream_k(c, o);
      DSF_HIP(launch_gemm(o, c.s));
    }
    return DSF_OK;
  }
  {  // h = x_kept + attn . W_o^T
    GemmArgs o = g;
    o.M = M; o.N = d; o.K = dq; o.K1 = dq;
    o.a = at<char>(c, c.plan.attn); o.lda = dq;
    o.b = W->w_o; o.ldb = dq;
    o.epi = EPI_RESID_STORE; o.bias = W->b_o;
    o.x = x; o.out = at<char>(c, c.plan.h); o.ldo = d;
    TimedScope ts(DSF_KIND_GEMM_O, c.s, true);
    use_stream_k(c, o);
    DSF_HIP(launch_gemm(o, c.s));
  }
  NormArgs n2{};
  n2.dtype = c.dtype;
  n2.src = at<char>(c, c.plan.h);
  n2.src_rows = 0;
  n2.B = B;
  n2.kk = kk;
  n2.d = d;
  n2.eps = D.norm_eps;
  n2.rms = 1;
  n2.w1 = W->norm2_w;
  n2.out1 = at<char>(c, c.plan.m2);
  DSF_HIP(launch_norm(n2, c.s));
  {  // SwiGLU: silu(gate) * up
    GemmArgs u = g;
    u.M = M; u.N = f; u.K = d; u.K1 = d;
    u.a = n2.out1; u.lda = d;
    u.b = W->w_up; u.ldb = d;
    u.epi = EPI_SWIGLU; u.f = f;
    u.out = at<char>(c, c.plan.act); u.ldo = f;
    TimedScope ts(DSF_KIND_GEMM_UP, c.s, true);
    use_stream_k(c, u);
    DSF_HIP(launch_gemm(u, c.s));
  }
  {  // y = h + act . W_down^T, scattered back
    GemmArgs o = g;
    o.M = M; o.N = d; o.K = f; o.K1 = f;
    o.a = at<char>(c, c.plan.act); o.lda = f;
    o.b = W->w_down; o.ldb = f;
    o.epi = gate ? EPI_RESID_SCATTER_GATE : EPI_RESID_SCATTER; o.bias = W->b_down;
    o.x = x; o.res = at<char>(c, c.plan.h); o.gate = scores;
    TimedScope ts(DSF_KIND_GEMM_DOWN, c.s, true);
    use_stream_k(c, o);
    DSF_HIP(launch_gemm(o, c.s));
  }
  return DSF_OK;
}

int check_common(const dsf_layer_desc* desc, int dtype, void* x, int B, int T, int k_max, int flags,
                 void* workspace, size_t workspace_bytes, bool with_sim, Plan* plan, bool with_align = false) {
  int rc = check_desc(desc);
  if (rc) return rc;
  rc = check_dtype(dtype);
  if (rc) return rc;
  DSF_CHECK(B >= 0 && T >= 0, DSF_EINVAL, "B and T must be >= 0");
  DSF_CHECK(int64_t(B) * T < (int64_t(1) << 31) / 8, DSF_EINVAL, "B * T too large");
  DSF_CHECK((flags & ~(DSF_FLAG_DENSE | DSF_FLAG_GATE)) == 0, DSF_EINVAL, "unknown flag bits 0x%x", flags);
  DSF_CHECK((flags & (DSF_FLAG_DENSE | DSF_FLAG_GATE)) != (DSF_FLAG_DENSE | DSF_FLAG_GATE), DSF_EINVAL,
            "DSF_FLAG_GATE needs router scores: it cannot be combined with DSF_FLAG_DENSE");
  if (B == 0 || T == 0 || k_max == 0) return DSF_OK;
  DSF_CHECK(x, DSF_EINVAL, "x is null");
  DSF_CHECK(aligned16(x), DSF_EINVAL, "x must be 16-byte aligned");
  *plan = make_plan(*desc, dtype, B, T, k_max, with_sim, with_align);
  DSF_CHECK(workspace_bytes >= plan->total, DSF_EWORKSPACE, "workspace needs %zu bytes, got %zu", plan->total,
            workspace_bytes);
  DSF_CHECK(workspace && (reinterpret_cast<uintptr_t>(workspace) & 255u) == 0, DSF_EINVAL,
            "workspace must be non-null and 256-byte aligned");
  return DSF_OK;
}
}  // namespace

extern "C" int dsf_sparse_block_forward(const dsf_layer_desc* desc, const dsf_layer_weights* weights, int dtype,
                                        void* x, int B, int T, int k, int flags, float* scores_out, int32_t* idx_out,
                                        const int32_t* idx_in, void* workspace, size_t workspace_bytes,
                                        hipStream_t stream) {
  DSF_CHECK(k >= 0 && k <= T, DSF_EINVAL, "k=%d outside [0, T=%d]", k, T);
  const bool dense = flags & DSF_FLAG_DENSE;
  DSF_CHECK(!dense || k == T, DSF_EINVAL, "DSF_FLAG_DENSE requires k == T");
  DSF_CHECK(!(dense && (scores_out || idx_out || idx_in)), DSF_EINVAL, "routing buffers are unused with DSF_FLAG_DENSE");
  Plan plan{};
  int rc = check_common(desc, dtype, x, B, T, k, flags, workspace, workspace_bytes, false, &plan);
  if (rc) return rc;
  if (B == 0 || T == 0 || k == 0) return DSF_OK;
  rc = check_weights(*desc, weights, 0);
  if (rc) return rc;
  rc = check_device();
  if (rc) return rc;
  Ctx c{desc, dtype, B, T, (char*)workspace, plan, stream, 0, nullptr};
  rc = get_aux(&c.aux);
  if (rc) return rc;
  rc = reset_stream_k(c);
  if (rc) return rc;
  DSF_HIP(launch_rope_table(at<float>(c, plan.rope), T, desc->rotary_dims, desc->rope_theta, stream));
  return run_layer(c, weights, x, k, dense, (flags & DSF_FLAG_GATE) != 0, scores_out, idx_out, idx_in);
}

extern "C" int dsf_stack_forward(const dsf_layer_desc* desc, const dsf_layer_weights* weights, int L, int dtype,
                                 const int* k, void* x, int B, int T, int flags, double* sim_accum, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream) {
  DSF_CHECK(L >= 0, DSF_EINVAL, "L < 0");
  DSF_CHECK(L == 0 || (weights && k), DSF_EINVAL, "null weights or k");
  const bool dense = flags & DSF_FLAG_DENSE;
  int k_max = 0;
  for (int l = 0; l < L; ++l) {
    DSF_CHECK(k[l] >= 0 && k[l] <= T, DSF_EINVAL, "k[%d]=%d outside [0, T=%d]", l, k[l], T);
    DSF_CHECK(!dense || k[l] == T, DSF_EINVAL, "DSF_FLAG_DENSE requires k[l] == T");
    k_max = k[l] > k_max ? k[l] : k_max;
  }
  const bool with_sim = sim_accum != nullptr;
  if (with_sim && L > 0 && B > 0 && T > 0) k_max = k_max > 1 ? k_max : 1;  // workspace for the input copy
  Plan plan{};
  int rc = check_common(desc, dtype, x, B, T, k_max, flags, workspace, workspace_bytes, with_sim, &plan);
  if (rc) return rc;
  if (L == 0 || B == 0 || T == 0 || k_max == 0) return DSF_OK;
  for (int l = 0; l < L; ++l) {
    rc = check_weights(*desc, &weights[l], l);
    if (rc) return rc;
  }
  rc = check_device();
  if (rc) return rc;
  Ctx c{desc, dtype, B, T, (char*)workspace, plan, stream, 0, nullptr};
  rc = get_aux(&c.aux);
  if (rc) return rc;
  rc = reset_stream_k(c);
  if (rc) return rc;
  DSF_HIP(launch_rope_table(at<float>(c, plan.rope), T, desc->rotary_dims, desc->rope_theta, stream));
  const size_t xbytes = elem_bytes(dtype) * size_t(B) * T * desc->d_model;
  for (int l = 0; l < L; ++l) {
    if (with_sim) DSF_HIP(launch_copy(x, at<char>(c, plan.xin), xbytes, stream));
    if (k[l] > 0) {
      rc = run_layer(c, &weights[l], x, k[l], dense, (flags & DSF_FLAG_GATE) != 0, nullptr, nullptr, nullptr);
      if (rc) return rc;
    }
    if (with_sim)
      DSF_HIP(launch_sim_stats(dtype, at<char>(c, plan.xin), x, int64_t(B) * T, desc->d_model, nullptr,
                               at<double>(c, plan.simpart), sim_accum + 2 * l, stream));
  }
  return DSF_OK;
}

// ------------------------------------------- incremental decoding

namespace {
// Size of the static scratch array of dsf_decode_step_static.
constexpr size_t kStaticScratchBytes = size_t(32) << 20;

struct DecodePlan {
  size_t scores, keep, gate, a1, a2, q, k, v, attn, act, h, m2, rope, part, spart, counters, total;
  size_t acount, scount;  // byte offsets within the counters block (zeroed together)
  int64_t ncounters;
};

DecodePlan make_decode_plan(const dsf_layer_desc& D, int dtype, int B, int max_pos, int cap) {
  const size_t eb = elem_bytes(dtype), n = size_t(B);
  const bool qwen = D.block == DSF_BLOCK_QWEN_SEQ;
  DecodePlan p{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += up256(bytes > 0 ? bytes : 1);
    return o;
  };
  p.scores = take(4 * n);
  p.keep = take(4 * n);
  p.gate = take(4 * n);
  p.a1 = take(eb * n * D.d_model);
  p.a2 = qwen ? 0 : take(eb * n * D.d_model);
  p.q = take(eb * n * D.n_heads * D.head_dim);
  p.k = take(eb * n * D.n_kv_heads * D.head_dim);
  p.v = take(eb * n * D.n_kv_heads * D.head_dim);
  p.attn = take(eb * n * D.n_heads * D.head_dim);
  p.act = take(eb * n * D.d_ff);
  p.h = qwen ? take(eb * n * D.d_model) : 0;
  p.m2 = qwen ? take(eb * n * D.d_model) : 0;
  p.rope = take(4 * size_t(max_pos) * D.rotary_dims);
  p.part = take(4 * n * D.n_heads * size_t(decode_attn_chunks(cap)) * (D.head_dim + 2));
  // few-row GEMMs (bf16, B <= 16): split-K partial tiles
  const bool few = dtype == DSF_BF16 && B <= 16;
  p.spart = few ? take(gemm_skinny_partial_bytes()) : 0;
  // counters, zero at the start of a step: decode attention (B * Hq chunk
  // counters, then B head counters), then the few-row GEMMs' tile counters
  const int64_t na = int64_t(n) * D.n_heads + n, ns = few ? gemm_skinny_counters() : 0;
  p.ncounters = na + ns;
  p.counters = take(sizeof(uint32_t) * size_t(p.ncounters));
  p.acount = p.counters;
  p.scount = few ? p.counters + sizeof(uint32_t) * size_t(na) : 0;
  p.total = off;
  return p;
}

struct DecCtx {
  const dsf_layer_desc* D;
  int dtype, B, max_pos, cap;
  char* ws;
  DecodePlan plan;
  hipStream_t s;
};

template <typename P>
P* dat(const DecCtx& c, size_t off) {
  return reinterpret_cast<P*>(c.ws + off);
}

// One layer of a decode step on the B new tokens (one row of x per sequence).
// Every row runs through the projections; the keep flags select which rows
// append to the cache and which receive the block's update (gate +inf / -inf
// in the gated residual epilogue: exactly x + delta or x).
int run_decode_layer(const DecCtx& c, const dsf_layer_weights* W, void* x, const int32_t* pos, const float* thr,
                     float* scores_out, int32_t* keep_out, void* ck, void* cv, int32_t* len) {
  const dsf_layer_desc& D = *c.D;
  const int B = c.B, d = D.d_model, hd = D.head_dim, Hq = D.n_heads, Hkv = D.n_kv_heads, f = D.d_ff;
  const int dq = Hq * hd, dkv = Hkv * hd;
  const bool qwen = D.block == DSF_BLOCK_QWEN_SEQ;
  float* scores = scores_out ? scores_out : dat<float>(c, c.plan.scores);
  int32_t* keep = dat<int32_t>(c, c.plan.keep);
  float* gate = dat<float>(c, c.plan.gate);
  const RouteArgs ra{thr, len, c.cap, keep, gate, keep_out};
  DSF_HIP(launch_router(c.dtype, x, B, d, D.d_router, W->router_w1, W->router_b1, W->router_w2, W->router_b2,
                        scores, c.s, &ra));

  NormArgs na{};
  na.dtype = c.dtype;
  na.src = x;
  na.src_rows = 0;  // compact rows: x [B, d]
  na.B = B;
  na.kk = 1;
  na.d = d;
  na.eps = D.norm_eps;
  na.rms = qwen;
  na.w1 = W->norm1_w;
  na.b1 = W->norm1_b;
  na.out1 = dat<char>(c, c.plan.a1);
  if (!qwen) {
    na.w2 = W->norm2_w;
    na.b2 = W->norm2_b;
    na.out2 = dat<char>(c, c.plan.a2);
  }
  DSF_HIP(launch_norm(na, c.s));

  GemmArgs g{};
  g.dtype = c.dtype;
  g.B = B;
  g.kk = 1;
  g.T = 1;
  g.M = B;
  if (c.plan.scount) {
    g.spart = dat<float>(c, c.plan.spart);
    g.scount = dat<uint32_t>(c, c.plan.scount);
  }
  if (!qwen) {  // FFN up + GELU on LN2
    GemmArgs u = g;
    u.N = f; u.K = d; u.K1 = d;
    u.a = na.out2; u.lda = d;
    u.b = W->w_up; u.ldb = d;
    u.epi = EPI_BIAS_GELU; u.bias = W->b_up;
    u.out = dat<char>(c, c.plan.act); u.ldo = f;
    DSF_HIP(launch_gemm(u, c.s));
  }
  {  // QKV, bias, RoPE at each new token's position
    GemmArgs q = g;
    q.T = c.max_pos;
    q.idx = pos;
    q.N = dq + 2 * dkv; q.K = d; q.K1 = d;
    q.a = na.out1; q.lda = d;
    q.b = W->w_qkv; q.ldb = d;
    q.epi = EPI_QKV_ROPE;
    q.bias = W->b_qkv;
    q.q = dat<char>(c, c.plan.q); q.k = dat<char>(c, c.plan.k); q.v = dat<char>(c, c.plan.v);
    q.Hq = Hq; q.Hkv = Hkv; q.hd = hd; q.R = D.rotary_dims;
    q.rope = dat<float>(c, c.plan.rope);
    DSF_HIP(launch_gemm(q, c.s));
  }
  // attention over the cache and the new token, appending the kept tokens' rows
  DSF_HIP(launch_decode_attention(c.dtype, dat<char>(c, c.plan.q), ck, cv, len, dat<char>(c, c.plan.k),
                                  dat<char>(c, c.plan.v), keep, B, Hq, Hkv, hd, c.cap, dat<float>(c, c.plan.part),
                                  dat<uint32_t>(c, c.plan.acount), dat<char>(c, c.plan.attn), c.s));
  if (!qwen) {  // parallel residual: [attn | act] . [W_o | W_down]^T + biases, gated by keep
    GemmArgs o = g;
    o.N = d; o.K = dq + f; o.K1 = dq;
    o.a = dat<char>(c, c.plan.attn); o.lda = dq;
    o.a2 = dat<char>(c, c.plan.act); o.lda2 = f;
    o.b = W->w_o; o.ldb = dq;
    o.b2 = W->w_down; o.ldb2 = f;
    o.epi = EPI_RESID_SCATTER_GATE; o.bias = W->b_o; o.bias2 = W->b_down;
    o.x = x; o.gate = gate;
    DSF_HIP(launch_gemm(o, c.s));
    return DSF_OK;
  }
  {  // h = x + attn . W_o^T
    GemmArgs o = g;
    o.N = d; o.K = dq; o.K1 = dq;
    o.a = dat<char>(c, c.plan.attn); o.lda = dq;
    o.b = W->w_o; o.ldb = dq;
    o.epi = EPI_RESID_STORE; o.bias = W->b_o;
    o.x = x; o.out = dat<char>(c, c.plan.h); o.ldo = d;
    DSF_HIP(launch_gemm(o, c.s));
  }
  NormArgs n2{};
  n2.dtype = c.dtype;
  n2.src = dat<char>(c, c.plan.h);
  n2.src_rows = 0;
  n2.B = B;
  n2.kk = 1;
  n2.d = d;
  n2.eps = D.norm_eps;
  n2.rms = 1;
  n2.w1 = W->norm2_w;
  n2.out1 = dat<char>(c, c.plan.m2);
  DSF_HIP(launch_norm(n2, c.s));
  {  // SwiGLU
    GemmArgs u = g;
    u.N = f; u.K = d; u.K1 = d;
    u.a = n2.out1; u.lda = d;
    u.b = W->w_up; u.ldb = d;
    u.epi = EPI_SWIGLU; u.f = f;
    u.out = dat<char>(c, c.plan.act); u.ldo = f;
    DSF_HIP(launch_gemm(u, c.s));
  }
  {  // x + keep * ((h - x) + act . W_down^T)
    GemmArgs o = g;
    o.N = d; o.K = f; o.K1 = f;
    o.a = dat<char>(c, c.plan.act); o.lda = f;
    o.b = W->w_down; o.ldb = f;
    o.epi = EPI_RESID_SCATTER_GATE; o.bias = W->b_down;
    o.x = x; o.res = dat<char>(c, c.plan.h); o.gate = gate;
    DSF_HIP(launch_gemm(o, c.s));
  }
  return DSF_OK;
}

int check_caches(void* const* cache_k, void* const* cache_v, int L) {
  DSF_CHECK(cache_k && cache_v, DSF_EINVAL, "null cache pointer arrays");
  for (int l = 0; l < L; ++l) {
    DSF_CHECK(cache_k[l] && cache_v[l], DSF_EINVAL, "null cache for layer %d", l);
    DSF_CHECK(aligned16(cache_k[l]) && aligned16(cache_v[l]), DSF_EINVAL, "caches of layer %d must be 16-byte aligned",
              l);
  }
  return DSF_OK;
}
}  // namespace

extern "C" size_t dsf_decode_workspace_size(const dsf_layer_desc* desc, int dtype, int B, int max_pos, int cap) {
  if (check_desc(desc) || check_dtype(dtype) || B < 0 || max_pos < 1 || cap < 1 || cap > kDecodeMaxCap) return 0;
  return make_decode_plan(*desc, dtype, B, max_pos, cap).total;
}

namespace {
// use_static: the caller passes no workspace and the step runs in the
// device's static scratch array (dsf_decode_step_static), which get_scratch()
// resolves after the argument checks.
int get_scratch(void** out);

int decode_step_impl(const dsf_layer_desc* desc, const dsf_layer_weights* weights, int L, int dtype, void* x, int B,
                     const int32_t* pos, int max_pos, const float* thr, float* scores_out, int32_t* keep_out,
                     void* const* cache_k, void* const* cache_v, int32_t* cache_len, int cap, bool use_static,
                     void* workspace, size_t workspace_bytes, hipStream_t stream) {
  int rc = check_desc(desc);
  if (rc) return rc;
  rc = check_dtype(dtype);
  if (rc) return rc;
  DSF_CHECK(L >= 0 && B >= 0, DSF_EINVAL, "L and B must be >= 0");
  DSF_CHECK(B <= (1 << 20), DSF_EINVAL, "B too large");
  DSF_CHECK(max_pos >= 1 && cap >= 1, DSF_EINVAL, "max_pos and cap must be >= 1");
  DSF_CHECK(cap <= kDecodeMaxCap, DSF_EUNSUPPORTED, "cache capacity %d above %d slots", cap, kDecodeMaxCap);
  DSF_CHECK(int64_t(B) * desc->n_kv_heads * cap * desc->head_dim < (int64_t(1) << 40), DSF_EINVAL, "cache too large");
  if (L == 0 || B == 0) return DSF_OK;
  DSF_CHECK(weights && x && pos && thr && cache_len, DSF_EINVAL, "null pointer");
  DSF_CHECK(aligned16(x), DSF_EINVAL, "x must be 16-byte aligned");
  rc = check_caches(cache_k, cache_v, L);
  if (rc) return rc;
  const DecodePlan plan = make_decode_plan(*desc, dtype, B, max_pos, cap);
  if (use_static) {
    DSF_CHECK(plan.total <= kStaticScratchBytes, DSF_EWORKSPACE,
              "this step needs %zu bytes of scratch, above the static scratch of %zu bytes (use dsf_decode_step "
              "with a workspace)", plan.total, kStaticScratchBytes);
  } else {
    DSF_CHECK(workspace_bytes >= plan.total, DSF_EWORKSPACE, "workspace needs %zu bytes, got %zu", plan.total,
              workspace_bytes);
    DSF_CHECK(workspace && (reinterpret_cast<uintptr_t>(workspace) & 255u) == 0, DSF_EINVAL,
              "workspace must be non-null and 256-byte aligned");
  }
  for (int l = 0; l < L; ++l) {
    rc = check_weights(*desc, &weights[l], l);
    if (rc) return rc;
  }
  rc = check_device();
  if (rc) return rc;
  if (use_static) {
    rc = get_scratch(&workspace);
    if (rc) return rc;
  }
  DecCtx c{desc, dtype, B, max_pos, cap, (char*)workspace, plan, stream};
  DSF_HIP(launch_rope_table(dat<float>(c, plan.rope), max_pos, desc->rotary_dims, desc->rope_theta, stream));
  DSF_HIP(launch_zero_u32(dat<uint32_t>(c, plan.counters), plan.ncounters, stream));
  for (int l = 0; l < L; ++l) {
    rc = run_decode_layer(c, &weights[l], x, pos, thr + size_t(l) * B, scores_out ? scores_out + size_t(l) * B : nullptr,
                          keep_out ? keep_out + size_t(l) * B : nullptr, cache_k[l], cache_v[l],
                          cache_len + size_t(l) * B);
    if (rc) return rc;
  }
  return DSF_OK;
}

// Static scratch of dsf_decode_step_static: one copy per device, loaded with
// the library's code object and held until the process ends. In host code
// `scratch` names a host-side stand-in, not device memory: its device address
// comes from hipGetSymbolAddress, once per device with that device current,
// and only that address is handed to kernels.
__device__ __align__(256) char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int get_scratch(void** out) {
  int dev = 0;
  DSF_HIP(hipGetDevice(&dev));
  DSF_CHECK(dev >= 0 && dev < kMaxDevices, DSF_EUNSUPPORTED, "device %d beyond the %d supported", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    DSF_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    DSF_CHECK(p && (reinterpret_cast<uintptr_t>(p) & 255u) == 0, DSF_EHIP, "static scratch has no usable address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return DSF_OK;
}
}  // namespace

extern "C" int dsf_decode_step(const dsf_layer_desc* desc, const dsf_layer_weights* weights, int L, int dtype,
                               void* x, int B, const int32_t* pos, int max_pos, const float* thr, float* scores_out,
                               int32_t* keep_out, void* const* cache_k, void* const* cache_v, int32_t* cache_len,
                               int cap, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return decode_step_impl(desc, weights, L, dtype, x, B, pos, max_pos, thr, scores_out, keep_out, cache_k, cache_v,
                          cache_len, cap, false, workspace, workspace_bytes, stream);
}

extern "C" size_t dsf_decode_static_scratch_bytes(void) { return kStaticScratchBytes; }

extern "C" int dsf_decode_step_static(const dsf_layer_desc* desc, const dsf_layer_weights* weights, int L,
                                      int dtype, void* x, int B, const int32_t* pos, int max_pos, const float* thr,
                                      float* scores_out, int32_t* keep_out, void* const* cache_k,
                                      void* const* cache_v, int32_t* cache_len, int cap, hipStream_t stream) {
  return decode_step_impl(desc, weights, L, dtype, x, B, pos, max_pos, thr, scores_out, keep_out, cache_k, cache_v,
                          cache_len, cap, true, nullptr, 0, stream);
}

extern "C" int dsf_stack_prefill(const dsf_layer_desc* desc, const dsf_layer_weights* weights, int L, int dtype,
                                 const int* k, void* x, int B, int T, void* const* cache_k, void* const* cache_v,
                                 int32_t* cache_len, int cap, float* thr_out, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream) {
  DSF_CHECK(L >= 0, DSF_EINVAL, "L < 0");
  DSF_CHECK(L == 0 || (weights && k), DSF_EINVAL, "null weights or k");
  DSF_CHECK(cap >= 1, DSF_EINVAL, "cap must be >= 1");
  int k_max = 0;
  for (int l = 0; l < L; ++l) {
    DSF_CHECK(k[l] >= 0 && k[l] <= T && k[l] <= cap, DSF_EINVAL, "k[%d]=%d outside [0, min(T=%d, cap=%d)]", l, k[l],
              T, cap);
    k_max = k[l] > k_max ? k[l] : k_max;
  }
  Plan plan{};
  int rc = check_common(desc, dtype, x, B, T, k_max, 0, workspace, workspace_bytes, false, &plan);
  if (rc) return rc;
  if (L == 0 || B == 0) return DSF_OK;
  DSF_CHECK(cache_len, DSF_EINVAL, "null cache_len");
  rc = check_caches(cache_k, cache_v, L);
  if (rc) return rc;
  for (int l = 0; l < L; ++l) {
    rc = check_weights(*desc, &weights[l], l);
    if (rc) return rc;
  }
  rc = check_device();
  if (rc) return rc;
  Ctx c{desc, dtype, B, T, (char*)workspace, plan, stream, 0, nullptr};
  rc = get_aux(&c.aux);
  if (rc) return rc;
  rc = reset_stream_k(c);
  if (rc) return rc;
  if (T > 0) DSF_HIP(launch_rope_table(at<float>(c, plan.rope), T, desc->rotary_dims, desc->rope_theta, stream));
  for (int l = 0; l < L; ++l) {
    if (k[l] > 0) {
      rc = run_layer(c, &weights[l], x, k[l], false, false, nullptr, nullptr, nullptr);
      if (rc) return rc;
    }
    DSF_HIP(launch_kv_fill(dtype, at<char>(c, plan.k), at<char>(c, plan.v), cache_k[l], cache_v[l],
                           cache_len + size_t(l) * B, B, desc->n_kv_heads, desc->head_dim, k[l], cap, stream));
    if (thr_out)
      DSF_HIP(launch_kept_min_score(at<float>(c, plan.scores), at<int32_t>(c, plan.idx), B, T, k[l],
                                    thr_out + size_t(l) * B, stream));
  }
  return DSF_OK;
}

// ------------------------------------------- alignment objective (Sec. 3.5)

extern "C" size_t dsf_align_workspace_size(int64_t n_rows) {
  if (n_rows < 0) return 0;
  return up256(sizeof(double) * size_t(n_rows > 0 ? n_rows : 1));
}

extern "C" int dsf_align_hidden(const void* h_sparse, const void* h_dense, int dtype, int64_t n_tokens, int d,
                                float* per_token_sq, double* accum, void* workspace, size_t workspace_bytes,
                                hipStream_t stream) {
  int rc = check_dtype(dtype);
  if (rc) return rc;
  DSF_CHECK(n_tokens >= 0 && n_tokens < (int64_t(1) << 40), DSF_EINVAL, "bad n_tokens");
  DSF_CHECK(d > 0 && d % 8 == 0 && d <= align_max_d(dtype), DSF_EUNSUPPORTED,
            "d must be a positive multiple of 8, at most %d for this dtype", align_max_d(dtype));
  if (n_tokens == 0) return DSF_OK;
  DSF_CHECK(h_sparse && h_dense && accum, DSF_EINVAL, "null pointer");
  DSF_CHECK(aligned16(h_sparse) && aligned16(h_dense), DSF_EINVAL, "hidden states must be 16-byte aligned");
  DSF_CHECK(workspace && workspace_bytes >= dsf_align_workspace_size(n_tokens), DSF_EWORKSPACE,
            "workspace needs %zu bytes", dsf_align_workspace_size(n_tokens));
  rc = check_device();
  if (rc) return rc;
  DSF_HIP(launch_align_hidden(dtype, h_sparse, h_dense, n_tokens, d, per_token_sq, (double*)workspace, accum,
                              stream));
  return DSF_OK;
}

extern "C" int dsf_kl_align(const void* logits_dense, const void* logits_sparse, int dtype, int64_t n_rows,
                            int n_classes, float* per_row_kl, double* accum, void* workspace, size_t workspace_bytes,
                            hipStream_t stream) {
  int rc = check_dtype(dtype);
  if (rc) return rc;
  DSF_CHECK(n_rows >= 0 && n_rows < (int64_t(1) << 31), DSF_EINVAL, "bad n_rows");
  DSF_CHECK(n_classes > 0 && n_classes % 8 == 0, DSF_EUNSUPPORTED, "n_classes must be a positive multiple of 8");
  if (n_rows == 0) return DSF_OK;
  DSF_CHECK(logits_dense && logits_sparse && accum, DSF_EINVAL, "null pointer");
  DSF_CHECK(aligned16(logits_dense) && aligned16(logits_sparse), DSF_EINVAL, "logits must be 16-byte aligned");
  DSF_CHECK(workspace && workspace_bytes >= dsf_align_workspace_size(n_rows), DSF_EWORKSPACE,
            "workspace needs %zu bytes", dsf_align_workspace_size(n_rows));
  rc = check_device();
  if (rc) return rc;
  DSF_HIP(launch_kl_align(dtype, logits_dense, logits_sparse, n_rows, n_classes, per_row_kl, (double*)workspace,
                          accum, stream));
  return DSF_OK;
}

extern "C" size_t dsf_align_stack_workspace_size(const dsf_layer_desc* desc, int dtype, int B, int T) {
  if (check_desc(desc) || check_dtype(dtype) || B < 0 || T < 0) return 0;
  if (desc->d_model > align_max_d(dtype)) return 0;
  return make_plan(*desc, dtype, B, T, T, false, true).total;
}

extern "C" int dsf_align_stack_forward(const dsf_layer_desc* desc, const dsf_layer_weights* weights, int L,
                                       int dtype, const int* k, void* x_sparse, void* x_dense, int B, int T,
                                       int flags, double* hid_accum, void* workspace, size_t workspace_bytes,
                                       hipStream_t stream) {
  DSF_CHECK(L >= 0, DSF_EINVAL, "L < 0");
  DSF_CHECK(L == 0 || (weights && k && hid_accum), DSF_EINVAL, "null weights, k or hid_accum");
  DSF_CHECK((flags & DSF_FLAG_DENSE) == 0, DSF_EINVAL, "the student cannot be dense (DSF_FLAG_DENSE)");
  for (int l = 0; l < L; ++l) DSF_CHECK(k[l] >= 0 && k[l] <= T, DSF_EINVAL, "k[%d]=%d outside [0, T=%d]", l, k[l], T);
  Plan plan{};
  int rc = check_common(desc, dtype, x_sparse, B, T, T, flags, workspace, workspace_bytes, false, &plan, true);
  if (rc) return rc;
  if (L == 0 || B == 0 || T == 0) return DSF_OK;
  DSF_CHECK(desc->d_model <= align_max_d(dtype), DSF_EUNSUPPORTED, "d_model above %d", align_max_d(dtype));
  DSF_CHECK(x_dense && aligned16(x_dense), DSF_EINVAL, "x_dense must be non-null and 16-byte aligned");
  for (int l = 0; l < L; ++l) {
    rc = check_weights(*desc, &weights[l], l);
    if (rc) return rc;
  }
  rc = check_device();
  if (rc) return rc;
  Ctx c{desc, dtype, B, T, (char*)workspace, plan, stream, 0, nullptr};
  rc = get_aux(&c.aux);
  if (rc) return rc;
  rc = reset_stream_k(c);
  if (rc) return rc;
  DSF_HIP(launch_rope_table(at<float>(c, plan.rope), T, desc->rotary_dims, desc->rope_theta, stream));
  const bool gate = (flags & DSF_FLAG_GATE) != 0;
  for (int l = 0; l < L; ++l) {
    rc = run_layer(c, &weights[l], x_dense, T, true, false, nullptr, nullptr, nullptr);  // teacher
    if (rc) return rc;
    if (k[l] > 0) {
      rc = run_layer(c, &weights[l], x_sparse, k[l], false, gate, nullptr, nullptr, nullptr);  // student
      if (rc) return rc;
    }
    DSF_HIP(launch_align_hidden(dtype, x_sparse, x_dense, int64_t(B) * T, desc->d_model, nullptr,
                                at<double>(c, plan.alignpart), hid_accum + l, stream));
  }
  return DSF_OK;
}

// ------------------------------ backward of the routed layer (Sec. 3.4)

namespace {
struct BwdPlan {
  size_t ctl, skpart, rope, xc, a1, a2, h, m2, q, k, v, attn, u, dd, du, dm, dao, dattn, dqf, dkf, dvf, lse, dvec, dqkv, da, acc;
  size_t mean1, rstd1, mean2, rstd2, wdT, wuT, woT, wqT, tdd, tact, tdu, tm, tdao, tattn, tdqkv, ta1, part, total;
  int Np, fup, dqkv_cols;
};

BwdPlan make_bwd_plan(const dsf_layer_desc& D, int B, int T, int k) {
  const size_t N = size_t(B) * k, d = D.d_model, dq = size_t(D.n_heads) * D.head_dim,
               dkv = size_t(D.n_kv_heads) * D.head_dim, f = D.d_ff;
  const bool qwen = D.block == DSF_BLOCK_QWEN_SEQ;
  BwdPlan p{};
  p.Np = int((N + 63) / 64 * 64);
  p.fup = int(qwen ? 2 * f : f);
  p.dqkv_cols = int(dq + 2 * dkv);
  const size_t Np = size_t(p.Np), fup = size_t(p.fup), cq = size_t(p.dqkv_cols);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += up256(bytes > 0 ? bytes : 1);
    return o;
  };
  // control block at offset 0 (status word, then the stream-K flags), as in
  // the forward's workspace, and the stream-K partial tiles
  p.ctl = take(sizeof(uint32_t) * (size_t(kCtlFlagsWord) + size_t(gemm_flag_count())));
  p.skpart = take(gemm_partial_bytes());
  p.rope = take(4 * size_t(T) * D.rotary_dims);
  p.xc = take(2 * N * d);
  p.a1 = take(2 * N * d);
  p.a2 = qwen ? 0 : take(2 * N * d);
  p.h = qwen ? take(2 * N * d) : 0;
  p.m2 = qwen ? take(2 * N * d) : 0;
  p.q = take(2 * N * dq);
  p.k = take(2 * N * dkv);
  p.v = take(2 * N * dkv);
  p.attn = take(2 * N * dq);
  p.u = take(2 * N * fup);
  p.dd = take(2 * N * d);
  p.du = take(2 * N * fup);
  p.dm = take(2 * N * d);
  p.dao = qwen ? take(2 * N * d) : p.dd;
  p.dattn = take(2 * N * dq);
  p.dqf = take(4 * N * dq);
  p.dkf = take(4 * N * dkv);
  p.dvf = take(4 * N * dkv);
  p.lse = take(4 * size_t(B) * D.n_heads * k);
  p.dvec = take(4 * size_t(B) * D.n_heads * k);
  p.dqkv = take(2 * N * cq);
  p.da = take(2 * N * d);
  p.acc = take(4 * N * d);
  p.mean1 = take(4 * N);
  p.rstd1 = take(4 * N);
  p.mean2 = take(4 * N);
  p.rstd2 = take(4 * N);
  p.wdT = take(2 * f * d);
  p.wuT = take(2 * d * fup);
  p.woT = take(2 * dq * d);
  p.wqT = take(2 * d * cq);
  p.tdd = take(2 * d * Np);
  p.tact = take(2 * f * Np);
  p.tdu = take(2 * fup * Np);
  p.tm = take(2 * d * Np);
  p.tdao = qwen ? take(2 * d * Np) : p.tdd;
  p.tattn = take(2 * dq * Np);
  p.tdqkv = take(2 * cq * Np);
  p.ta1 = take(2 * d * Np);
  const size_t cmax = std::max(std::max(d, fup), cq);
  p.part = take(4 * size_t(colsum_chunks(int(N))) * cmax);
  p.total = off;
  return p;
}

int check_bwd(const dsf_layer_desc* desc, int dtype, int B, int T, int k) {
  int rc = check_desc(desc);
  if (rc) return rc;
  DSF_CHECK(dtype == DSF_BF16, DSF_EUNSUPPORTED, "the layer backward is provided for DSF_BF16 only");
  DSF_CHECK(B >= 0 && T >= 0 && k >= 0 && k <= T, DSF_EINVAL, "need B, T >= 0 and k in [0, T]");
  DSF_CHECK(int64_t(B) * T < (int64_t(1) << 31) / 8, DSF_EINVAL, "B * T too large");
  return DSF_OK;
}

// The stream-K state of one backward call: partial tiles, flags and status
// word in its workspace, and the last epoch handed out since the flags were
// zeroed.
struct BwdSk {
  float* part;
  uint32_t *flags, *status;
  uint32_t epoch;
};

// C[M, N] = A[M, K] . Bm[N, K]^T with one of the backward epilogues (plain
// token rows: no positions, one "sequence" of M rows). With sk, a launch may
// take the stream-K grid (the weight gradients, whose few output tiles would
// leave most of the chip idle while each reduces over every kept token).
int bwd_gemm(int epi, int M, int N, int K, const void* A, int lda, const void* Bm, int ldb, void* out, int ldo,
             const void* bias, const void* res, int f, hipStream_t s, BwdSk* sk = nullptr) {
  if (M == 0 || N == 0) return DSF_OK;
  GemmArgs g{};
  g.dtype = DSF_BF16;
  g.M = M; g.N = N; g.K = K; g.K1 = K;
  g.a = A; g.lda = lda; g.b = Bm; g.ldb = ldb;
  g.epi = epi; g.bias = bias; g.res = res; g.f = f;
  g.out = out; g.ldo = ldo;
  g.B = 1; g.kk = M; g.T = M;
  if (sk) {
    g.part = sk->part;
    g.flags = sk->flags;
    g.status = sk->status;
    g.epoch = ++sk->epoch;
  }
  DSF_HIP(launch_gemm(g, s));
  return DSF_OK;
}
}  // namespace

extern "C" size_t dsf_backward_workspace_size(const dsf_layer_desc* desc, int dtype, int B, int T, int k) {
  if (check_bwd(desc, dtype, B, T, k)) return 0;
  return make_bwd_plan(*desc, B, T, k).total;
}

extern "C" int dsf_sparse_block_backward(const dsf_layer_desc* desc, const dsf_layer_weights* weights, int dtype,
                                         const void* x, const void* dy, int B, int T, int k, const int32_t* idx,
                                         const float* scores, int flags, void* dx, const dsf_layer_grads* grads,
                                         void* workspace, size_t workspace_bytes, hipStream_t stream) {
  int rc = check_bwd(desc, dtype, B, T, k);
  if (rc) return rc;
  DSF_CHECK((flags & ~DSF_FLAG_GATE) == 0, DSF_EINVAL, "only DSF_FLAG_GATE is accepted (flags 0x%x)", flags);
  const bool gate = flags & DSF_FLAG_GATE;
  if (B == 0 || T == 0) return DSF_OK;
  DSF_CHECK(x && dy && dx, DSF_EINVAL, "null x, dy or dx");
  DSF_CHECK(aligned16(x) && aligned16(dy) && aligned16(dx), DSF_EINVAL, "x, dy and dx must be 16-byte aligned");
  DSF_CHECK(k == 0 || idx, DSF_EINVAL, "null idx");
  DSF_CHECK(!gate || scores, DSF_EINVAL, "DSF_FLAG_GATE needs the router scores");
  rc = check_weights(*desc, weights, 0);
  if (rc) return rc;
  static const dsf_layer_grads kNone{};
  const dsf_layer_grads& G = grads ? *grads : kNone;
  const float* gp[] = {G.w_qkv, G.b_qkv, G.w_o, G.b_o, G.w_up, G.b_up, G.w_down, G.b_down,
                       G.norm1_w, G.norm1_b, G.norm2_w, G.norm2_b};
  for (const float* p : gp) DSF_CHECK(aligned16(p), DSF_EINVAL, "gradient buffers must be 16-byte aligned");
  const dsf_layer_desc& D = *desc;
  const bool qwen = D.block == DSF_BLOCK_QWEN_SEQ;
  const BwdPlan p = make_bwd_plan(D, B, T, k);
  DSF_CHECK(workspace_bytes >= p.total, DSF_EWORKSPACE, "workspace needs %zu bytes, got %zu", p.total,
            workspace_bytes);
  DSF_CHECK(workspace && (reinterpret_cast<uintptr_t>(workspace) & 255u) == 0, DSF_EINVAL,
            "workspace must be non-null and 256-byte aligned");
  rc = check_device();
  if (rc) return rc;
  hipStream_t s = stream;
  char* ws = (char*)workspace;
  // zero the control block: the status word and the stream-K flags
  BwdSk sk{reinterpret_cast<float*>(ws + p.skpart), reinterpret_cast<uint32_t*>(ws + p.ctl) + kCtlFlagsWord,
           reinterpret_cast<uint32_t*>(ws + p.ctl), 0};
  DSF_HIP(launch_zero_u32(sk.status, int64_t(kCtlFlagsWord) + gemm_flag_count(), s));
  const size_t xbytes = size_t(B) * T * D.d_model * 2;
  DSF_HIP(launch_copy(dy, dx, xbytes, s));  // skipped rows: dx = dy
  if (k == 0) return DSF_OK;                // (the weight gradients are then not written)
  auto P = [&](size_t off) { return (void*)(ws + off); };
  auto F = [&](size_t off) { return (float*)(ws + off); };
  const int d = D.d_model, hd = D.head_dim, Hq = D.n_heads, Hkv = D.n_kv_heads, f = D.d_ff;
  const int dq = Hq * hd, dkv = Hkv * hd, N = B * k, Np = p.Np, fup = p.fup, cq = p.dqkv_cols;

  // ---- recompute the forward's activations of the kept rows
  DSF_HIP(launch_rope_table(F(p.rope), T, D.rotary_dims, D.rope_theta, s));
  DSF_HIP(launch_gather(dtype, x, B, T, d, idx, k, P(p.xc), s));
  NormArgs na{};
  na.dtype = dtype; na.src = P(p.xc); na.src_rows = 0; na.B = B; na.kk = k; na.d = d; na.eps = D.norm_eps;
  na.rms = qwen; na.w1 = weights->norm1_w; na.b1 = weights->norm1_b; na.out1 = P(p.a1);
  if (!qwen) {
    na.w2 = weights->norm2_w; na.b2 = weights->norm2_b; na.out2 = P(p.a2);
  }
  DSF_HIP(launch_norm(na, s));
  {
    GemmArgs g{};
    g.dtype = dtype; g.B = B; g.kk = k; g.T = T; g.idx = idx;
    g.M = N; g.N = dq + 2 * dkv; g.K = d; g.K1 = d;
    g.a = P(p.a1); g.lda = d; g.b = weights->w_qkv; g.ldb = d;
    g.epi = EPI_QKV_ROPE; g.bias = weights->b_qkv;
    g.q = P(p.q); g.k = P(p.k); g.v = P(p.v);
    g.Hq = Hq; g.Hkv = Hkv; g.hd = hd; g.R = D.rotary_dims; g.rope = F(p.rope);
    DSF_HIP(launch_gemm(g, s));
  }
  DSF_HIP(launch_attention(dtype, P(p.q), P(p.k), P(p.v), B, Hq, Hkv, k, hd, P(p.attn), s, F(p.lse)));
  const void* mrows;  // input rows of the up projection
  if (!qwen) {
    mrows = P(p.a2);
    rc = bwd_gemm(EPI_STORE, N, f, d, P(p.a2), d, weights->w_up, d, P(p.u), f, weights->b_up, nullptr, 0, s);
    if (rc) return rc;
  } else {
    GemmArgs g{};  // h = x_kept + attn W_o^T
    g.dtype = dtype; g.B = B; g.kk = k; g.T = T; g.idx = idx;
    g.M = N; g.N = d; g.K = dq; g.K1 = dq;
    g.a = P(p.attn); g.lda = dq; g.b = weights->w_o; g.ldb = dq;
    g.epi = EPI_RESID_STORE; g.bias = weights->b_o;
    g.x = const_cast<void*>(x); g.out = P(p.h); g.ldo = d;
    DSF_HIP(launch_gemm(g, s));
    NormArgs n2{};
    n2.dtype = dtype; n2.src = P(p.h); n2.src_rows = 0; n2.B = B; n2.kk = k; n2.d = d; n2.eps = D.norm_eps;
    n2.rms = 1; n2.w1 = weights->norm2_w; n2.out1 = P(p.m2);
    DSF_HIP(launch_norm(n2, s));
    mrows = P(p.m2);
    rc = bwd_gemm(EPI_STORE, N, 2 * f, d, P(p.m2), d, weights->w_up, d, P(p.u), 2 * f, nullptr, nullptr, 0, s);
    if (rc) return rc;
  }

  // ---- the adjoint: d(delta) = gate * dy at the kept rows
  DSF_HIP(launch_gather_scale(dy, B, T, d, idx, k, gate ? scores : nullptr, P(p.dd), s));
  // FFN down projection
  if (G.w_down) {
    DSF_HIP(launch_transpose(0, P(p.dd), N, d, d, P(p.tdd), Np, s));
    DSF_HIP(launch_transpose(qwen ? 2 : 1, P(p.u), N, f, fup, P(p.tact), Np, s));
    rc = bwd_gemm(EPI_STORE_F32, d, f, Np, P(p.tdd), Np, P(p.tact), Np, G.w_down, f, nullptr, nullptr, 0, s, &sk);
    if (rc) return rc;
  }
  if (G.b_down && !qwen) DSF_HIP(launch_colsum(P(p.dd), N, d, d, nullptr, nullptr, nullptr, F(p.part), G.b_down, s));
  DSF_HIP(launch_transpose(0, weights->w_down, d, f, f, P(p.wdT), d, s));
  rc = bwd_gemm(qwen ? EPI_SWIGLU_BWD : EPI_GELU_BWD, N, f, d, P(p.dd), d, P(p.wdT), d, P(p.du), fup, nullptr, P(p.u),
                f, s);
  if (rc) return rc;
  // FFN up projection
  if (G.w_up) {
    DSF_HIP(launch_transpose(0, P(p.du), N, fup, fup, P(p.tdu), Np, s));
    DSF_HIP(launch_transpose(0, mrows, N, d, d, P(p.tm), Np, s));
    rc = bwd_gemm(EPI_STORE_F32, fup, d, Np, P(p.tdu), Np, P(p.tm), Np, G.w_up, d, nullptr, nullptr, 0, s, &sk);
    if (rc) return rc;
  }
  if (G.b_up && !qwen) DSF_HIP(launch_colsum(P(p.du), N, f, f, nullptr, nullptr, nullptr, F(p.part), G.b_up, s));
  DSF_HIP(launch_transpose(0, weights->w_up, fup, d, d, P(p.wuT), fup, s));
  rc = bwd_gemm(EPI_STORE, N, d, fup, P(p.du), fup, P(p.wuT), fup, P(p.dm), d, nullptr, nullptr, 0, s);
  if (rc) return rc;
  // second norm: NeoX's LN2 of the kept rows, Qwen's RMS2 of h = x + attention
  if (!qwen) {
    DSF_HIP(launch_norm_bwd(false, P(p.xc), P(p.dm), weights->norm2_w, N, d, D.norm_eps, F(p.acc), false, nullptr,
                            nullptr, F(p.mean2), F(p.rstd2), s));
  } else {
    DSF_HIP(launch_norm_bwd(true, P(p.h), P(p.dm), weights->norm2_w, N, d, D.norm_eps, F(p.acc), false, P(p.dd),
                            P(p.dao), F(p.mean2), F(p.rstd2), s));
  }
  if (G.norm2_w)
    DSF_HIP(launch_colsum(P(p.dm), N, d, d, qwen ? P(p.h) : P(p.xc), qwen ? nullptr : F(p.mean2), F(p.rstd2),
                          F(p.part), G.norm2_w, s));
  if (G.norm2_b && !qwen) DSF_HIP(launch_colsum(P(p.dm), N, d, d, nullptr, nullptr, nullptr, F(p.part), G.norm2_b, s));
  // attention output projection
  if (G.w_o) {
    if (qwen || !G.w_down) DSF_HIP(launch_transpose(0, P(p.dao), N, d, d, P(p.tdao), Np, s));
    DSF_HIP(launch_transpose(0, P(p.attn), N, dq, dq, P(p.tattn), Np, s));
    rc = bwd_gemm(EPI_STORE_F32, d, dq, Np, P(p.tdao), Np, P(p.tattn), Np, G.w_o, dq, nullptr, nullptr, 0, s, &sk);
    if (rc) return rc;
  }
  if (G.b_o && !qwen) DSF_HIP(launch_colsum(P(p.dao), N, d, d, nullptr, nullptr, nullptr, F(p.part), G.b_o, s));
  DSF_HIP(launch_transpose(0, weights->w_o, d, dq, dq, P(p.woT), d, s));
  rc = bwd_gemm(EPI_STORE, N, dq, d, P(p.dao), d, P(p.woT), d, P(p.dattn), dq, nullptr, nullptr, 0, s);
  if (rc) return rc;
  // attention over the kept tokens, then RoPE turned back into token-major dqkv
  DSF_HIP(launch_attention_bwd(P(p.q), P(p.k), P(p.v), P(p.attn), P(p.dattn), B, Hq, Hkv, k, hd, F(p.lse),
                               F(p.dvec), F(p.dqf), F(p.dkf), F(p.dvf), s));
  DSF_HIP(launch_rope_bwd(F(p.dqf), F(p.dkf), F(p.dvf), F(p.rope), idx, B, k, T, Hq, Hkv, hd, D.rotary_dims,
                          P(p.dqkv), s));
  // QKV projection
  if (G.w_qkv) {
    DSF_HIP(launch_transpose(0, P(p.dqkv), N, cq, cq, P(p.tdqkv), Np, s));
    DSF_HIP(launch_transpose(0, P(p.a1), N, d, d, P(p.ta1), Np, s));
    rc = bwd_gemm(EPI_STORE_F32, cq, d, Np, P(p.tdqkv), Np, P(p.ta1), Np, G.w_qkv, d, nullptr, nullptr, 0, s, &sk);
    if (rc) return rc;
  }
  if (G.b_qkv) DSF_HIP(launch_colsum(P(p.dqkv), N, cq, cq, nullptr, nullptr, nullptr, F(p.part), G.b_qkv, s));
  DSF_HIP(launch_transpose(0, weights->w_qkv, cq, d, d, P(p.wqT), cq, s));
  rc = bwd_gemm(EPI_STORE, N, d, cq, P(p.dqkv), cq, P(p.wqT), cq, P(p.da), d, nullptr, nullptr, 0, s);
  if (rc) return rc;
  // first norm of the kept rows
  DSF_HIP(launch_norm_bwd(qwen, P(p.xc), P(p.da), weights->norm1_w, N, d, D.norm_eps, F(p.acc), true, nullptr,
                          nullptr, F(p.mean1), F(p.rstd1), s));
  if (G.norm1_w)
    DSF_HIP(launch_colsum(P(p.da), N, d, d, P(p.xc), qwen ? nullptr : F(p.mean1), F(p.rstd1), F(p.part), G.norm1_w,
                          s));
  if (G.norm1_b && !qwen) DSF_HIP(launch_colsum(P(p.da), N, d, d, nullptr, nullptr, nullptr, F(p.part), G.norm1_b, s));
  // kept rows: dx = dy + the block's gradient (the residual path carries dy)
  DSF_HIP(launch_scatter_grad(dy, F(p.acc), B, T, d, idx, k, dx, s));
  return DSF_OK;
}
