// Host side of libmls: argument validation, workspace planning and the launch
// sequence of the forward and backward passes (C ABI declared in mls.h).
//
// Forward:  fused tile kernel (partials) -> label logits -> row merge -> mean.
// Backward: h_i^T once; then per vocabulary chunk of Vc rows:
//           W_i[chunk]^T -> fused dlogits tile kernel (slab G, G^T)
//           -> grad_W_i[chunk] = G^T h_i -> grad_h_i += G W_i[chunk].
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <string>
#include <vector>

#include "mls.h"
#include "mls_launch.h"

namespace {

using namespace mls;

thread_local std::string g_last_error;

// Per-thread kernel timing (mls_profile_enable / mls_profile_report).
struct ProfRec {
  const char* name;
  hipEvent_t start;
  hipEvent_t stop;
};
struct Profiler {
  bool on = false;
  std::vector<ProfRec> recs;
  std::vector<hipEvent_t> pool;
  hipEvent_t take() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
};
thread_local Profiler g_prof;

// Brackets one kernel launch with events when profiling is on.
struct ProfScope {
  hipStream_t s;
  ProfRec rec{nullptr, nullptr, nullptr};
  ProfScope(const char* name, hipStream_t st) : s(st) {
    if (!g_prof.on) return;
    rec.name = name;
    rec.start = g_prof.take();
    rec.stop = g_prof.take();
    if (rec.start && rec.stop) hipEventRecord(rec.start, s);
  }
  ~ProfScope() {
    if (!rec.name || !rec.start || !rec.stop) return;
    hipEventRecord(rec.stop, s);
    g_prof.recs.push_back(rec);
  }
};

mls_status fail(mls_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

mls_status hip_fail(hipError_t e, const char* what) {
  return fail(MLS_HIP_ERROR, "%s: %s", what, hipGetErrorString(e));
}

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

constexpr int64_t kSlabTargetBytes = 4ll << 30;  // logit-gradient slab(s) per chunk
constexpr int64_t kMinChunks = 4;                 // the default plan never holds a [T, V] slab
constexpr int64_t kRecordBudget = 1ll << 30;      // forward partial records of one token chunk
constexpr int64_t kLogitSlabBudget = 16ll << 30;  // stored logits of one token chunk (all sub-models)
constexpr int64_t kPanelMax = (1ll << 32) - 1;    // bytes one wide-GEMM operand may span

struct Plan {
  int M = 0;
  int s = 0;
  bool f32 = false;
  bool wide = false;  // wide bf16 tile core (every width a multiple of 64)
  int es = 2;
  int64_t T = 0, V = 0;
  int64_t sumd = 0;
  int64_t T_pad = 0;
  int n_tt = 0;
  int n_vt_fwd = 0;
  // forward token chunks: the partial records of one chunk at a time
  int64_t fwd_tc = 0;
  int fwd_nc = 0;
  // fused forward + backward (mls_distill_fwd_bwd): with fb_store, token chunks
  // of fb_tc rows whose logits are stored (fp16, row length fb_ld) and turned
  // into the logit gradient in place; otherwise the forward, then the
  // recompute backward
  bool fb_store = false;
  int64_t fb_tc = 0;
  int fb_nc = 0;
  int64_t fb_ld = 0;
  size_t fb_off_lslab = 0, fb_off_part = 0, fb_off_lab = 0, fb_bytes = 0;
  int64_t Vc = 0;
  int n_chunks = 0;
  // The wide gradient GEMM addresses its M-contiguous operands (the slab,
  // h_i, the head chunk) with 32-bit offsets over the whole K extent, so each
  // must stay below 4 GiB; a backward where h_i alone would not takes the
  // general path, which addresses with 64 bits.
  bool wide_bwd = false;
  // forward workspace
  size_t off_partials = 0, off_lab = 0, fwd_bytes = 0;
  // backward workspace (off_ghp: fp32 partial sums of a bf16 grad_h over vocabulary chunks)
  bool grad_h_bf16 = false;
  size_t off_slab = 0, off_slabT = 0, off_hT = 0, off_WT = 0, off_ghp = 0, bwd_bytes = 0;
  // diagnostics workspace (vocabulary segments of the pairwise pass)
  int n_vt_diag = 0, n_tt_diag = 0;
  int m_diag = 0;  // sub-models per diagnostics pass (at most kMaxDiagModels)
  size_t off_dpart = 0, off_drow = 0, off_dsub = 0, off_dam = 0, diag_bytes = 0;
  size_t ws_bytes = 0;
  size_t stats_bytes = 0;
  size_t header_off = 0;
};

mls_status validate(const mls_problem* p) {
  if (!p) return fail(MLS_INVALID_ARG, "problem is NULL");
  if (p->M < 1 || p->M > MLS_MAX_MODELS)
    return fail(MLS_INVALID_ARG, "M=%d outside [1, %d]", p->M, MLS_MAX_MODELS);
  if (p->teacher < -1 || p->teacher >= p->M)
    return fail(MLS_INVALID_ARG, "teacher=%d outside [-1, M)", p->teacher);
  if (p->T < 1 || p->T > (1ll << 30)) return fail(MLS_INVALID_ARG, "T=%lld out of range", (long long)p->T);
  if (p->V < 2 || p->V > (1ll << 30)) return fail(MLS_INVALID_ARG, "V=%lld out of range", (long long)p->V);
  if (p->in_dtype != MLS_BF16 && p->in_dtype != MLS_F32)
    return fail(MLS_UNSUPPORTED, "in_dtype=%d unsupported", p->in_dtype);
  if (p->grad_h_dtype != MLS_BF16 && p->grad_h_dtype != MLS_F32)
    return fail(MLS_UNSUPPORTED, "grad_h_dtype=%d unsupported", p->grad_h_dtype);
  if (!(p->tau > 0.0f) || !isfinite(p->tau)) return fail(MLS_INVALID_ARG, "tau must be finite and > 0");
  if (!isfinite(p->alpha) || p->alpha < 0.0f || p->alpha > 1.0f)
    return fail(MLS_INVALID_ARG, "alpha must be in [0, 1]");
  if (p->vocab_chunk < 0) return fail(MLS_INVALID_ARG, "vocab_chunk must be >= 0");
  if (!p->labels) return fail(MLS_INVALID_ARG, "labels is NULL");
  if (!aligned(p->labels, 8)) return fail(MLS_INVALID_ARG, "labels not 8-byte aligned");
  const int64_t gran = p->in_dtype == MLS_BF16 ? 8 : 4;
  for (int i = 0; i < p->M; ++i) {
    if (p->d[i] < 1 || p->d[i] > (1 << 20))
      return fail(MLS_INVALID_ARG, "d[%d]=%lld out of range", i, (long long)p->d[i]);
    if (p->d[i] % gran)
      return fail(MLS_UNSUPPORTED, "d[%d]=%lld is not a multiple of %lld", i, (long long)p->d[i],
                  (long long)gran);
    if (!p->h[i] || !p->W[i]) return fail(MLS_INVALID_ARG, "h[%d] or W[%d] is NULL", i, i);
    if (!aligned(p->h[i], 16) || !aligned(p->W[i], 16))
      return fail(MLS_INVALID_ARG, "h[%d] or W[%d] not 16-byte aligned", i, i);
  }
  return MLS_OK;
}

void make_plan(const mls_problem* p, Plan& pl) {
  pl.M = p->M;
  pl.s = p->teacher < 0 ? p->M - 1 : p->teacher;
  pl.f32 = p->in_dtype == MLS_F32;
  pl.es = pl.f32 ? 4 : 2;
  pl.T = p->T;
  pl.V = p->V;
  pl.sumd = 0;
  for (int i = 0; i < p->M; ++i) pl.sumd += p->d[i];
  pl.wide = !pl.f32;
  for (int i = 0; i < p->M; ++i) pl.wide = pl.wide && (p->d[i] % 64 == 0);
  pl.T_pad = round_up(p->T, kFusedBN);
  pl.n_tt = (int)(pl.T_pad / kFusedBN);
  const int fbm = fused_tile_rows(pl.wide);
  pl.n_vt_fwd = (int)((p->V + fbm - 1) / fbm);
  int64_t dmax = 0;
  for (int i = 0; i < p->M; ++i) dmax = std::max<int64_t>(dmax, p->d[i]);
  pl.wide_bwd = pl.wide && pl.T_pad * dmax * pl.es <= kPanelMax && pl.T_pad * 256 * pl.es <= kPanelMax;
  const int64_t vmax = round_up(p->V, 256);
  int64_t vc;
  if (p->vocab_chunk > 0) {
    vc = round_up(p->vocab_chunk, 256);
  } else {
    // At least kMinChunks balanced chunks, more when the slabs of one chunk
    // would exceed kSlabTargetBytes (the wide path keeps one slab layout, the
    // general path two), so the logit-gradient slab never spans the whole
    // vocabulary (V > 256).
    const int64_t per_row = (pl.wide_bwd ? 1ll : 2ll) * pl.M * pl.T_pad * pl.es;
    const int64_t fit = std::max<int64_t>(256, kSlabTargetBytes / per_row / 256 * 256);
    const int64_t n = std::max<int64_t>(kMinChunks, (p->V + fit - 1) / fit);
    vc = round_up((p->V + n - 1) / n, 256);
  }
  if (pl.wide_bwd) {
    // one slab [T_pad][Vc] and one head chunk [Vc][d_i] below 4 GiB each
    const int64_t cap = std::min(kPanelMax / (pl.T_pad * pl.es), kPanelMax / (dmax * pl.es)) / 256 * 256;
    vc = std::min(vc, cap);
  }
  pl.Vc = std::max<int64_t>(256, std::min(vc, vmax));
  pl.n_chunks = (int)((p->V + pl.Vc - 1) / pl.Vc);
  pl.grad_h_bf16 = p->grad_h_dtype == MLS_BF16;

  // forward: token chunks whose partial records stay within kRecordBudget
  const int64_t rec_per_tok = (int64_t)pl.M * pl.n_vt_fwd * kFusedFwdParts * (int64_t)sizeof(float4);
  pl.fwd_tc = std::min<int64_t>(pl.T_pad, std::max<int64_t>(kFusedBN, kRecordBudget / rec_per_tok /
                                                                          kFusedBN * kFusedBN));
  pl.fwd_nc = (int)((p->T + pl.fwd_tc - 1) / pl.fwd_tc);
  size_t off = 0;
  pl.off_partials = off;
  off = align256(off + (size_t)rec_per_tok * pl.fwd_tc);
  pl.off_lab = off;
  off = align256(off + (size_t)pl.M * pl.T * sizeof(float));
  pl.fwd_bytes = off;

  off = 0;
  const size_t slab = (size_t)pl.M * pl.T_pad * pl.Vc * pl.es;
  pl.off_slab = off;
  off = align256(off + slab);
  if (!pl.wide_bwd) {  // general path: G^T slab and transposed operands as well
    pl.off_slabT = off;
    off = align256(off + slab);
    pl.off_hT = off;
    off = align256(off + (size_t)pl.sumd * pl.T_pad * pl.es);
    pl.off_WT = off;
    off = align256(off + (size_t)pl.sumd * pl.Vc * pl.es);
  }
  if (pl.grad_h_bf16 && pl.n_chunks > 1) {
    pl.off_ghp = off;
    off = align256(off + (size_t)pl.sumd * pl.T * sizeof(float));
  }
  pl.bwd_bytes = off;

  // diagnostics: one record per (vocabulary tile, token) of the sub-models of
  // one pass; suites of more than kMaxDiagModels run several passes over
  // subsets, each staged and scattered into the outputs
  {
    const int md = std::min(pl.M, kMaxDiagModels);
    pl.m_diag = md;
    pl.n_vt_diag = (int)((p->V + diag_tile_rows(pl.wide) - 1) / diag_tile_rows(pl.wide));
    pl.n_tt_diag = (int)((p->T + diag_tile_cols(pl.wide, md) - 1) / diag_tile_cols(pl.wide, md));
    off = 0;
    pl.off_dpart = off;
    off = align256(off + (size_t)pl.n_vt_diag * kDiagParts * pl.T * diag_record_floats(md) *
                             sizeof(float));
    pl.off_drow = off;
    off = align256(off + (size_t)pl.T * 2 * md * md * sizeof(float));
    if (pl.M > kMaxDiagModels) {
      pl.off_dsub = off;
      off = align256(off + 2 * kMaxDiagModels * kMaxDiagModels * sizeof(float));
      pl.off_dam = off;
      off = align256(off + (size_t)kMaxDiagModels * pl.T * sizeof(int32_t));
    }
    pl.diag_bytes = off;
  }
  pl.ws_bytes = std::max(std::max(pl.fwd_bytes, pl.bwd_bytes), pl.diag_bytes);

  // fused forward + backward with stored logits: at least two token chunks (so
  // no [T, V] logits exist), each sub-model's fp16 slab below 4 GiB (the wide
  // GEMM's 32-bit offsets) and all of them within kLogitSlabBudget; every head
  // [V, d_i] must also fit one wide-GEMM operand
  pl.fb_ld = (int64_t)pl.n_vt_fwd * kFusedBN;
  const bool heads_fit = pl.V * dmax * pl.es <= kPanelMax;
  pl.fb_store = pl.wide && p->T > kFusedBN && heads_fit && !(p->flags & MLS_FWD_BWD_RECOMPUTE);
  if (pl.fb_store) {
    const int64_t row = pl.fb_ld * 2;
    int64_t cap = std::min<int64_t>(kPanelMax / row, kLogitSlabBudget / (row * pl.M));
    cap = cap / kFusedBN * kFusedBN;
    if (cap < kFusedBN) {
      pl.fb_store = false;
    } else {
      const int64_t n = std::max<int64_t>(2, (p->T + cap - 1) / cap);
      pl.fb_tc = round_up((p->T + n - 1) / n, kFusedBN);
      pl.fb_nc = (int)((p->T + pl.fb_tc - 1) / pl.fb_tc);
    }
  }
  if (pl.fb_store) {
    off = 0;
    pl.fb_off_lslab = off;
    off = align256(off + (size_t)pl.M * pl.fb_tc * pl.fb_ld * 2);
    pl.fb_off_part = off;
    off = align256(off + (size_t)rec_per_tok * pl.fb_tc);
    pl.fb_off_lab = off;
    off = align256(off + (size_t)pl.M * pl.T * sizeof(float));
    pl.fb_bytes = off;
  } else {
    pl.fb_bytes = std::max(pl.fwd_bytes, pl.bwd_bytes);
  }

  pl.header_off = (size_t)(4ll * pl.M * pl.T + pl.T) * sizeof(float);
  pl.stats_bytes = align256(pl.header_off + 2 * sizeof(int32_t));
}

void fill_order(const Plan& pl, int32_t* order) {
  int k = 0;
  order[k++] = pl.s;
  for (int i = 0; i < pl.M; ++i)
    if (i != pl.s) order[k++] = i;
  for (; k < kMaxModels; ++k) order[k] = 0;
}

void fill_common(const mls_problem* p, const Plan& pl, FusedArgs& a) {
  memset(&a, 0, sizeof(a));
  a.M = pl.M;
  a.teacher = pl.s;
  fill_order(pl, a.order);
  for (int i = 0; i < pl.M; ++i) {
    a.h[i] = p->h[i];
    a.W[i] = p->W[i];
    a.d[i] = p->d[i];
  }
  a.T = pl.T;
  a.V = pl.V;
  a.labels = p->labels;
  a.ignore_index = p->ignore_index;
  a.tau = p->tau;
  a.inv_tau = 1.0f / p->tau;
  a.wide = pl.wide ? 1 : 0;
  // vocabulary tiles per group of the tile order: measured best at 8 for
  // T <= 4096 and at 4 from T = 8192 on (V = 128,256 and 262,144 shapes)
  a.group_v = pl.n_tt >= 64 ? 4 : 8;
  a.n_tt = pl.n_tt;
  a.T_pad = pl.T_pad;
  a.Vc = pl.Vc;
}

void fill_rows(const mls_problem* p, const Plan& pl, RowArgs& r) {
  memset(&r, 0, sizeof(r));
  r.M = pl.M;
  r.teacher = pl.s;
  for (int i = 0; i < pl.M; ++i) {
    r.h[i] = p->h[i];
    r.W[i] = p->W[i];
    r.d[i] = p->d[i];
  }
  r.T = pl.T;
  r.V = pl.V;
  r.labels = p->labels;
  r.ignore_index = p->ignore_index;
  r.tau = p->tau;
  r.n_rec = pl.n_vt_fwd * kFusedFwdParts;
  fill_order(pl, r.order);
}

void host_coeffs(int M, int s, float alpha, float tau, int mode, const float* w, float* g_ce,
                 float* g_kl) {
  for (int i = 0; i < M; ++i) {
    const float wi = w ? w[i] : 1.0f;
    if (i == s) {
      g_ce[i] = wi;
      g_kl[i] = 0.0f;
    } else if (mode == MLS_MODE_PAPER) {
      g_ce[i] = wi * (1.0f - alpha);
      g_kl[i] = wi * alpha * tau * tau;
    } else {
      g_ce[i] = wi;
      g_kl[i] = wi * alpha * tau * tau;
    }
  }
}

// Label logits of every token and, when `count` is set, the valid-token count
// into the statistics header (which the logit-gradient pass reads before the
// loss mean is taken).
hipError_t launch_labels(const mls_problem* p, const Plan& pl, float* lab, void* stats, bool count,
                         hipStream_t s) {
  RowArgs r;
  fill_rows(p, pl, r);
  r.lab = lab;
  r.header = reinterpret_cast<int32_t*>(static_cast<char*>(stats) + pl.header_off);
  hipError_t e;
  {
    ProfScope ps("label_logits", s);
    e = launch_label_logits(r, pl.f32, s);
  }
  if (e != hipSuccess || !count) return e;
  ProfScope ps("count_valid", s);
  return launch_count_valid(r, s);
}

// Forward of tokens [t0, t0 + tc): the tile kernel (partial records, and with
// lslab the fp16 logits) and the row merge into the statistics.
hipError_t forward_chunk(const mls_problem* p, const Plan& pl, int64_t t0, int64_t tc,
                         float4* partials, const float* lab, uint16_t* lslab, void* stats,
                         hipStream_t s) {
  FusedArgs a;
  fill_common(p, pl, a);
  for (int i = 0; i < pl.M; ++i)
    a.h[i] = static_cast<const char*>(p->h[i]) + (size_t)t0 * p->d[i] * pl.es;
  a.T = tc;
  a.n_tt = (int)((tc + kFusedBN - 1) / kFusedBN);
  // vocabulary tiles per group of the tile order, measured per token chunk:
  // 8 at 16 token tiles over 393 vocabulary tiles (2,048-token chunks at
  // V = 50,304; 4 and 16 are 5 % slower), 4 at 32 token tiles over 1,002
  // vocabulary tiles (4,096-token chunks at V = 128,256; 5 % faster than 8)
  // and at 64 (8,192-token chunks, 1 %), level at 52 over 2,048 (6,656-token
  // chunks at V = 262,144)
  a.group_v = (a.n_tt >= 64 || (a.n_tt >= 32 && pl.n_vt_fwd >= 512)) ? 4 : 8;
  a.n_vt = pl.n_vt_fwd;
  a.partials = partials;
  a.lslab = lslab;
  a.ld_lslab = pl.fb_ld;
  hipError_t e;
  {
    ProfScope ps("fused_fwd", s);
    e = launch_fused_fwd(a, pl.f32, s);
  }
  if (e != hipSuccess) return e;
  RowArgs r;
  fill_rows(p, pl, r);
  r.t0 = t0;
  r.Tc = tc;
  r.partials = partials;
  r.lab = const_cast<float*>(lab);
  r.stats = static_cast<float*>(stats);
  ProfScope ps("row_merge", s);
  return launch_finalize_rows(r, s);
}

// Means over the valid tokens, the valid count and the device flags.
hipError_t finish_losses(const mls_problem* p, const Plan& pl, void* stats, float* ce, float* kl,
                         float* entropy, hipStream_t s) {
  RowArgs r;
  fill_rows(p, pl, r);
  r.stats = static_cast<float*>(stats);
  r.header = reinterpret_cast<int32_t*>(static_cast<char*>(stats) + pl.header_off);
  r.ce = ce;
  r.kl = kl;
  r.entropy = entropy;
  ProfScope ps("loss_mean", s);
  return launch_reduce_losses(r, s);
}

}  // namespace

namespace mls {
mls_status set_error(mls_status s, const char* what, const char* detail) {
  return fail(s, detail && detail[0] ? "%s: %s" : "%s%s", what, detail ? detail : "");
}
}  // namespace mls

extern "C" {

const char* mls_version(void) { return "mls 0.1.0 (gfx950)"; }

mls_status mls_device_info(int32_t* compute_units, int32_t* clock_khz, int32_t* mem_clock_khz,
                           int32_t* mem_bus_bits) {
  g_last_error.clear();
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  struct Q {
    int32_t* out;
    hipDeviceAttribute_t attr;
  } qs[] = {{compute_units, hipDeviceAttributeMultiprocessorCount},
            {clock_khz, hipDeviceAttributeClockRate},
            {mem_clock_khz, hipDeviceAttributeMemoryClockRate},
            {mem_bus_bits, hipDeviceAttributeMemoryBusWidth}};
  for (const Q& q : qs) {
    if (!q.out) continue;
    int v = 0;
    if ((e = hipDeviceGetAttribute(&v, q.attr, dev)) != hipSuccess)
      return hip_fail(e, "hipDeviceGetAttribute");
    *q.out = v;
  }
  return MLS_OK;
}

const char* mls_last_error(void) { return g_last_error.c_str(); }

const char* mls_status_string(mls_status s) {
  switch (s) {
    case MLS_OK: return "ok";
    case MLS_INVALID_ARG: return "invalid argument";
    case MLS_UNSUPPORTED: return "unsupported";
    case MLS_WORKSPACE_TOO_SMALL: return "workspace too small";
    case MLS_HIP_ERROR: return "HIP error";
  }
  return "unknown status";
}

mls_status mls_query_sizes(const mls_problem* p, size_t* workspace_bytes, size_t* stats_bytes) {
  g_last_error.clear();
  mls_status st = validate(p);
  if (st != MLS_OK) return st;
  Plan pl;
  make_plan(p, pl);
  if (workspace_bytes) *workspace_bytes = pl.ws_bytes;
  if (stats_bytes) *stats_bytes = pl.stats_bytes;
  return MLS_OK;
}

mls_status mls_coeffs(int32_t M, int32_t teacher, float alpha, float tau, int32_t mode,
                      const float* w, float* g_ce, float* g_kl) {
  g_last_error.clear();
  if (M < 1 || M > MLS_MAX_MODELS) return fail(MLS_INVALID_ARG, "M=%d outside [1, %d]", M, MLS_MAX_MODELS);
  if (teacher < -1 || teacher >= M) return fail(MLS_INVALID_ARG, "teacher=%d outside [-1, M)", teacher);
  if (!g_ce || !g_kl) return fail(MLS_INVALID_ARG, "output pointer is NULL");
  if (mode != MLS_MODE_PAPER && mode != MLS_MODE_ADDITIVE)
    return fail(MLS_INVALID_ARG, "unknown mode %d", mode);
  if (!(tau > 0.0f) || !isfinite(tau)) return fail(MLS_INVALID_ARG, "tau must be finite and > 0");
  if (!isfinite(alpha) || alpha < 0.0f || alpha > 1.0f) return fail(MLS_INVALID_ARG, "alpha must be in [0, 1]");
  host_coeffs(M, teacher < 0 ? M - 1 : teacher, alpha, tau, mode, w, g_ce, g_kl);
  return MLS_OK;
}

mls_status mls_distill_fwd(const mls_problem* p, void* stats, float* ce, float* kl, float* entropy,
                           void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  mls_status st = validate(p);
  if (st != MLS_OK) return st;
  if (!stats || !ce || !kl || !workspace)
    return fail(MLS_INVALID_ARG, "stats, ce, kl and workspace must be non-NULL");
  if (!aligned(stats, 16) || !aligned(workspace, 16) || !aligned(ce, 4) || !aligned(kl, 4))
    return fail(MLS_INVALID_ARG, "misaligned stats / workspace / loss pointer");
  Plan pl;
  make_plan(p, pl);
  if (workspace_bytes < pl.fwd_bytes)
    return fail(MLS_WORKSPACE_TOO_SMALL, "forward needs %zu workspace bytes, got %zu", pl.fwd_bytes,
                workspace_bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  float* lab = reinterpret_cast<float*>(ws + pl.off_lab);
  hipError_t e = launch_labels(p, pl, lab, stats, false, s);
  if (e != hipSuccess) return hip_fail(e, "label logits launch");
  for (int c = 0; c < pl.fwd_nc; ++c) {
    const int64_t t0 = (int64_t)c * pl.fwd_tc;
    e = forward_chunk(p, pl, t0, std::min(pl.fwd_tc, pl.T - t0),
                      reinterpret_cast<float4*>(ws + pl.off_partials), lab, nullptr, stats, s);
    if (e != hipSuccess) return hip_fail(e, "forward launch");
  }
  e = finish_losses(p, pl, stats, ce, kl, entropy, s);
  if (e != hipSuccess) return hip_fail(e, "loss reduction launch");
  return MLS_OK;
}

mls_status mls_distill_bwd(const mls_problem* p, const void* stats, const float* g_ce,
                           const float* g_kl, void* const* grad_h, float* const* grad_W,
                           void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  mls_status st = validate(p);
  if (st != MLS_OK) return st;
  if (!stats || !workspace || !grad_h || !grad_W)
    return fail(MLS_INVALID_ARG, "stats, workspace, grad_h and grad_W must be non-NULL");
  if ((g_ce == nullptr) != (g_kl == nullptr))
    return fail(MLS_INVALID_ARG, "g_ce and g_kl must both be given or both be NULL");
  if (!aligned(stats, 16) || !aligned(workspace, 16))
    return fail(MLS_INVALID_ARG, "misaligned stats / workspace");
  for (int i = 0; i < p->M; ++i) {
    if ((grad_h[i] && !aligned(grad_h[i], p->grad_h_dtype == MLS_BF16 ? 2 : 4)) ||
        (grad_W[i] && !aligned(grad_W[i], 4)))
      return fail(MLS_INVALID_ARG, "misaligned gradient pointer %d", i);
  }
  Plan pl;
  make_plan(p, pl);
  if (workspace_bytes < pl.bwd_bytes)
    return fail(MLS_WORKSPACE_TOO_SMALL, "backward needs %zu workspace bytes, got %zu", pl.bwd_bytes,
                workspace_bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  const float* sf = static_cast<const float*>(stats);

  FusedArgs a;
  fill_common(p, pl, a);
  a.wide = pl.wide_bwd ? 1 : 0;
  a.n_vt = (int)(pl.Vc / fused_tile_rows(pl.wide_bwd));
  a.lse1 = sf;
  a.lset = sf + (int64_t)pl.M * pl.T;
  a.n_valid = reinterpret_cast<const int32_t*>(static_cast<const char*>(stats) + pl.header_off);
  a.g_ce = g_ce;
  a.g_kl = g_kl;
  host_coeffs(pl.M, pl.s, p->alpha, p->tau, MLS_MODE_PAPER, nullptr, a.host_gce, a.host_gkl);
  a.slab = ws + pl.off_slab;
  a.slabT = pl.wide_bwd ? nullptr : ws + pl.off_slabT;
  char* hT = ws + pl.off_hT;
  char* WT = ws + pl.off_WT;

  int64_t doff[kMaxModels];
  int64_t acc = 0;
  for (int i = 0; i < pl.M; ++i) {
    doff[i] = acc;
    acc += p->d[i];
  }
  const size_t slab_stride = (size_t)pl.T_pad * pl.Vc * pl.es;
  const int tbm = gemm_tile_rows(pl.wide_bwd);
  const int tbn = gemm_tile_cols(pl.wide_bwd);
  hipError_t e;

  // general path: h_i^T [d_i, T_pad] for the grad_W products
  if (!pl.wide_bwd) {
    TransposeArgs ta;
    memset(&ta, 0, sizeof(ta));
    int64_t maxc = 0;
    for (int i = 0; i < pl.M; ++i) {
      if (!grad_W[i]) continue;
      TransposeJob& j = ta.j[ta.njobs++];
      j.src = p->h[i];
      j.dst = hT + (size_t)doff[i] * pl.T_pad * pl.es;
      j.ld_src = p->d[i];
      j.ld_dst = pl.T_pad;
      j.r0 = 0;
      j.src_rows = pl.T;
      j.out_rows = pl.T_pad;
      j.cols = p->d[i];
      maxc = std::max(maxc, p->d[i]);
    }
    {
      ProfScope ps("transpose_h", s);
      e = launch_transpose(ta, pl.T_pad, maxc, pl.f32, s);
    }
    if (e != hipSuccess) return hip_fail(e, "transpose launch");
  }

  for (int c = 0; c < pl.n_chunks; ++c) {
    const int64_t v0 = (int64_t)c * pl.Vc;
    const int64_t vrows = std::min(pl.Vc, pl.V - v0);

    // general path: W_i[chunk]^T [d_i, Vc] for the grad_h products
    if (!pl.wide_bwd) {
    TransposeArgs ta;
    memset(&ta, 0, sizeof(ta));
    int64_t maxc = 0;
    for (int i = 0; i < pl.M; ++i) {
      if (!grad_h[i]) continue;
      TransposeJob& j = ta.j[ta.njobs++];
      j.src = p->W[i];
      j.dst = WT + (size_t)doff[i] * pl.Vc * pl.es;
      j.ld_src = p->d[i];
      j.ld_dst = pl.Vc;
      j.r0 = v0;
      j.src_rows = pl.V;
      j.out_rows = pl.Vc;
      j.cols = p->d[i];
      maxc = std::max(maxc, p->d[i]);
    }
    {
      ProfScope ps("transpose_W", s);
      e = launch_transpose(ta, pl.Vc, maxc, pl.f32, s);
    }
    if (e != hipSuccess) return hip_fail(e, "transpose launch");
    }

    a.v0 = v0;
    if (pl.wide_bwd) {
      // The wide GEMM reads slab columns past the chunk's rows only up to the
      // K-tile holding its last row (grad_h) or for output rows it does not
      // store (grad_W), so the vocabulary tiles past the chunk end are skipped.
      const int bm = fused_tile_rows(true);
      if (bm % gemm_wide_k_tile() == 0) a.n_vt = (int)((vrows + bm - 1) / bm);
    }
    {
      ProfScope ps("fused_bwd", s);
      e = launch_fused_bwd(a, pl.f32, s);
    }
    if (e != hipSuccess) return hip_fail(e, "fused backward launch");

    // grad_h_i (+)= G_i W_i[chunk] and grad_W_i[chunk] = G_i^T h_i in one grouped
    // launch (the longer grad_h tiles first). The wide path reads the slab, the
    // head chunk and h in their stored layouts; the general path reads G^T and
    // the transposed operands.
    GemmArgs ga;
    memset(&ga, 0, sizeof(ga));
    int tiles = 0;
    for (int i = 0; i < pl.M; ++i) {
      if (!grad_h[i]) continue;
      GemmGroup& g = ga.g[ga.ngroups++];
      g.A = static_cast<const char*>(a.slab) + (size_t)i * slab_stride;
      g.lda = pl.Vc;
      g.rows = pl.T;
      if (pl.wide_bwd) {
        g.B = static_cast<const char*>(p->W[i]) + (size_t)v0 * p->d[i] * pl.es;  // [v][d]
        g.ldb = p->d[i];
        g.cols = vrows;
      } else {
        g.B = WT + (size_t)doff[i] * pl.Vc * pl.es;
        g.ldb = pl.Vc;
        g.cols = p->d[i];
      }
      // grad_h: fp32 output accumulated over the chunks; a bf16 output keeps the
      // partial sums of the earlier chunks in fp32 and is stored once, by the last
      const bool last = c == pl.n_chunks - 1;
      const bool acc_flag = (p->flags & MLS_ACCUMULATE_GRAD_H) != 0;
      float* ghp = pl.grad_h_bf16 && pl.n_chunks > 1
                       ? reinterpret_cast<float*>(ws + pl.off_ghp) + doff[i] * pl.T
                       : nullptr;
      if (!pl.grad_h_bf16) {
        g.C = static_cast<float*>(grad_h[i]);
        g.accumulate = (c > 0 || acc_flag) ? 1 : 0;
      } else if (!last) {
        g.C = ghp;
        g.accumulate = c > 0 ? 1 : 0;
      } else {
        g.Cb = static_cast<uint16_t*>(grad_h[i]);
        g.Cpart = ghp;
        g.accumulate = acc_flag ? 1 : 0;
      }
      g.ldc = p->d[i];
      g.ldc_rows = pl.T;
      // the chunk's rows past vrows read as zero from the head: the last,
      // shorter chunk stops at the K-tile holding its last row
      const int64_t kt = gemm_wide_k_tile();
      g.K = pl.wide_bwd ? std::min(pl.Vc, (vrows + kt - 1) / kt * kt) : pl.Vc;
      g.kind = 0;
      g.tiles_m = (int)((pl.T + tbm - 1) / tbm);
      g.tiles_n = (int)((p->d[i] + tbn - 1) / tbn);
      g.tile_begin = tiles;
      g.group_m = 8;
      tiles += g.tiles_m * g.tiles_n;
    }
    const int grad_h_tiles = tiles;
    for (int i = 0; i < pl.M; ++i) {
      if (!grad_W[i]) continue;
      GemmGroup& g = ga.g[ga.ngroups++];
      if (pl.wide_bwd) {
        g.A = static_cast<const char*>(a.slab) + (size_t)i * slab_stride;  // [t][v]
        g.lda = pl.Vc;
        g.rows = pl.T_pad;
        g.B = p->h[i];  // [t][d]
        g.ldb = p->d[i];
        g.cols = pl.T;
      } else {
        g.A = static_cast<const char*>(a.slabT) + (size_t)i * slab_stride;
        g.lda = pl.T_pad;
        g.rows = vrows;
        g.B = hT + (size_t)doff[i] * pl.T_pad * pl.es;
        g.ldb = pl.T_pad;
        g.cols = p->d[i];
      }
      g.C = grad_W[i] + v0 * p->d[i];
      g.ldc = p->d[i];
      g.ldc_rows = vrows;
      g.K = pl.T_pad;
      g.kind = 1;
      g.tiles_m = (int)((vrows + tbm - 1) / tbm);
      g.tiles_n = (int)((p->d[i] + tbn - 1) / tbn);
      g.tile_begin = tiles;
      g.accumulate = (p->flags & MLS_ACCUMULATE_GRAD_W) ? 1 : 0;
      g.group_m = 0;
      tiles += g.tiles_m * g.tiles_n;
    }
    // spread both phases evenly over the XCDs when every XCD's share of the
    // first phase fits in its block count
    ga.phase_tiles = 0;
    if (grad_h_tiles > 0 && grad_h_tiles < tiles) {
      bool fits = true;
      for (int x = 0; x < 8; ++x) {
        const int q1 = grad_h_tiles / 8 + (x < grad_h_tiles % 8 ? 1 : 0);
        if (q1 > (tiles - x + 7) / 8) fits = false;
      }
      if (fits) ga.phase_tiles = grad_h_tiles;
    }
    {
      ProfScope ps("gemm_grads", s);
      e = pl.wide_bwd ? launch_gemm_wide(ga, tiles, s) : launch_gemm_nt(ga, tiles, pl.f32, s);
    }
    if (e != hipSuccess) return hip_fail(e, "gradient GEMM launch");
  }
  return MLS_OK;
}

mls_status mls_query_fwd_bwd_workspace(const mls_problem* p, size_t* workspace_bytes) {
  g_last_error.clear();
  mls_status st = validate(p);
  if (st != MLS_OK) return st;
  if (!workspace_bytes) return fail(MLS_INVALID_ARG, "workspace_bytes is NULL");
  Plan pl;
  make_plan(p, pl);
  *workspace_bytes = pl.fb_bytes;
  return MLS_OK;
}

mls_status mls_distill_fwd_bwd(const mls_problem* p, void* stats, float* ce, float* kl,
                               float* entropy, const float* g_ce, const float* g_kl,
                               void* const* grad_h, float* const* grad_W, void* workspace,
                               size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  mls_status st = validate(p);
  if (st != MLS_OK) return st;
  if (!stats || !ce || !kl || !workspace || !grad_h || !grad_W)
    return fail(MLS_INVALID_ARG, "stats, ce, kl, workspace, grad_h and grad_W must be non-NULL");
  if ((g_ce == nullptr) != (g_kl == nullptr))
    return fail(MLS_INVALID_ARG, "g_ce and g_kl must both be given or both be NULL");
  if (!aligned(stats, 16) || !aligned(workspace, 16) || !aligned(ce, 4) || !aligned(kl, 4))
    return fail(MLS_INVALID_ARG, "misaligned stats / workspace / loss pointer");
  for (int i = 0; i < p->M; ++i) {
    if ((grad_h[i] && !aligned(grad_h[i], p->grad_h_dtype == MLS_BF16 ? 2 : 4)) ||
        (grad_W[i] && !aligned(grad_W[i], 4)))
      return fail(MLS_INVALID_ARG, "misaligned gradient pointer %d", i);
  }
  Plan pl;
  make_plan(p, pl);
  if (workspace_bytes < pl.fb_bytes)
    return fail(MLS_WORKSPACE_TOO_SMALL, "forward + backward needs %zu workspace bytes, got %zu",
                pl.fb_bytes, workspace_bytes);
  if (!pl.fb_store) {
    // one token tile, widths off the wide path, or the recompute plan asked for
    st = mls_distill_fwd(p, stats, ce, kl, entropy, workspace, workspace_bytes, stream);
    if (st != MLS_OK) return st;
    return mls_distill_bwd(p, stats, g_ce, g_kl, grad_h, grad_W, workspace, workspace_bytes, stream);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  float* lab = reinterpret_cast<float*>(ws + pl.fb_off_lab);
  float4* part = reinterpret_cast<float4*>(ws + pl.fb_off_part);
  uint16_t* lslab = reinterpret_cast<uint16_t*>(ws + pl.fb_off_lslab);
  hipError_t e = launch_labels(p, pl, lab, stats, true, s);
  if (e != hipSuccess) return hip_fail(e, "label logits launch");

  GradArgs ga;
  memset(&ga, 0, sizeof(ga));
  ga.M = pl.M;
  fill_order(pl, ga.order);
  ga.T = pl.T;
  ga.V = pl.V;
  ga.ld = pl.fb_ld;
  ga.labels = p->labels;
  ga.ignore_index = p->ignore_index;
  ga.inv_tau = 1.0f / p->tau;
  const float* sf = static_cast<const float*>(stats);
  ga.lse1 = sf;
  ga.lset = sf + (int64_t)pl.M * pl.T;
  ga.n_valid = reinterpret_cast<const int32_t*>(static_cast<const char*>(stats) + pl.header_off);
  ga.g_ce = g_ce;
  ga.g_kl = g_kl;
  host_coeffs(pl.M, pl.s, p->alpha, p->tau, MLS_MODE_PAPER, nullptr, ga.host_gce, ga.host_gkl);
  ga.partials = part;
  ga.n_rec = pl.n_vt_fwd * kFusedFwdParts;
  ga.slab = lslab;

  const int64_t kt = gemm_wide_k_tile();
  const int tbm = gemm_tile_rows(true);
  const int tbn = gemm_tile_cols(true);
  for (int c = 0; c < pl.fb_nc; ++c) {
    const int64_t t0 = (int64_t)c * pl.fb_tc;
    const int64_t tc = std::min(pl.fb_tc, pl.T - t0);
    const int64_t tc_pad = round_up(tc, kFusedBN);
    e = forward_chunk(p, pl, t0, tc, part, lab, lslab, stats, s);
    if (e != hipSuccess) return hip_fail(e, "forward launch");

    ga.Tc = tc;
    ga.Tc_pad = tc_pad;
    ga.t0 = t0;
    {
      ProfScope ps("grad_logits", s);
      e = launch_grad_logits(ga, s);
    }
    if (e != hipSuccess) return hip_fail(e, "logit gradient launch");

    // grad_h_i[chunk rows] = G_i W_i (K = V, complete in this chunk) and
    // grad_W_i (+)= G_i^T h_i[chunk rows] (K = the chunk's tokens), one launch
    const size_t slab_stride = (size_t)tc_pad * pl.fb_ld * 2;
    GemmArgs gm;
    memset(&gm, 0, sizeof(gm));
    int tiles = 0;
    for (int i = 0; i < pl.M; ++i) {
      if (!grad_h[i]) continue;
      GemmGroup& g = gm.g[gm.ngroups++];
      g.A = reinterpret_cast<const char*>(lslab) + (size_t)i * slab_stride;  // [t][v]
      g.lda = pl.fb_ld;
      g.rows = tc;
      g.B = p->W[i];  // [v][d]
      g.ldb = p->d[i];
      g.cols = pl.V;
      if (pl.grad_h_bf16)
        g.Cb = static_cast<uint16_t*>(grad_h[i]) + t0 * p->d[i];
      else
        g.C = static_cast<float*>(grad_h[i]) + t0 * p->d[i];
      g.accumulate = (p->flags & MLS_ACCUMULATE_GRAD_H) ? 1 : 0;
      g.ldc = p->d[i];
      g.ldc_rows = tc;
      g.K = round_up(pl.V, kt);
      g.kind = 0;
      g.tiles_m = (int)((tc + tbm - 1) / tbm);
      g.tiles_n = (int)((p->d[i] + tbn - 1) / tbn);
      g.tile_begin = tiles;
      g.group_m = 8;
      tiles += g.tiles_m * g.tiles_n;
    }
    const int grad_h_tiles = tiles;
    for (int i = 0; i < pl.M; ++i) {
      if (!grad_W[i]) continue;
      GemmGroup& g = gm.g[gm.ngroups++];
      g.A = reinterpret_cast<const char*>(lslab) + (size_t)i * slab_stride;  // [t][v] as [k][m]
      g.lda = pl.fb_ld;
      g.rows = tc_pad;
      g.B = static_cast<const char*>(p->h[i]) + (size_t)t0 * p->d[i] * pl.es;  // [t][d]
      g.ldb = p->d[i];
      g.cols = tc;
      g.C = grad_W[i];
      g.ldc = p->d[i];
      g.ldc_rows = pl.V;
      g.K = tc_pad;
      g.kind = 1;
      g.tiles_m = (int)((pl.V + tbm - 1) / tbm);
      g.tiles_n = (int)((p->d[i] + tbn - 1) / tbn);
      g.tile_begin = tiles;
      g.accumulate = (c > 0 || (p->flags & MLS_ACCUMULATE_GRAD_W)) ? 1 : 0;
      g.group_m = 0;
      tiles += g.tiles_m * g.tiles_n;
    }
    gm.phase_tiles = 0;
    if (grad_h_tiles > 0 && grad_h_tiles < tiles) {
      bool fits = true;
      for (int x = 0; x < 8; ++x) {
        const int q1 = grad_h_tiles / 8 + (x < grad_h_tiles % 8 ? 1 : 0);
        if (q1 > (tiles - x + 7) / 8) fits = false;
      }
      if (fits) gm.phase_tiles = grad_h_tiles;
    }
    {
      ProfScope ps("gemm_grads", s);
      e = launch_gemm_wide(gm, tiles, s);
    }
    if (e != hipSuccess) return hip_fail(e, "gradient GEMM launch");
  }
  e = finish_losses(p, pl, stats, ce, kl, entropy, s);
  if (e != hipSuccess) return hip_fail(e, "loss reduction launch");
  return MLS_OK;
}

mls_status mls_diagnostics(const mls_problem* p, float* kl_pair, float* agree, int32_t* argmax,
                           void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  mls_status st = validate(p);
  if (st != MLS_OK) return st;
  if (!kl_pair || !agree || !workspace)
    return fail(MLS_INVALID_ARG, "kl_pair, agree and workspace must be non-NULL");
  if (!aligned(workspace, 16) || !aligned(kl_pair, 4) || !aligned(agree, 4) || !aligned(argmax, 4))
    return fail(MLS_INVALID_ARG, "misaligned workspace / output pointer");
  Plan pl;
  make_plan(p, pl);
  if (workspace_bytes < pl.diag_bytes)
    return fail(MLS_WORKSPACE_TOO_SMALL, "diagnostics need %zu workspace bytes, got %zu",
                pl.diag_bytes, workspace_bytes);
  char* ws = static_cast<char*>(workspace);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // Passes: the whole suite, or subsets of kMaxDiagModels sub-models chosen
  // greedily (each adds the most pairs not yet covered) until every pair of
  // sub-models has shared a pass (a pair's KL and agreement need both logits).
  int subsets[64][kMaxDiagModels];
  int n_pass = 0;
  if (pl.M <= kMaxDiagModels) {
    for (int i = 0; i < pl.M; ++i) subsets[0][i] = i;
    n_pass = 1;
  } else {
    bool covered[kMaxModels][kMaxModels] = {};
    for (;;) {
      int best[kMaxDiagModels] = {0, 1, 2, 3}, best_gain = 0;
      int c[kMaxDiagModels];
      for (c[0] = 0; c[0] < pl.M; ++c[0])
        for (c[1] = c[0] + 1; c[1] < pl.M; ++c[1])
          for (c[2] = c[1] + 1; c[2] < pl.M; ++c[2])
            for (c[3] = c[2] + 1; c[3] < pl.M; ++c[3]) {
              int gain = 0;
              for (int x = 0; x < kMaxDiagModels; ++x)
                for (int y = x + 1; y < kMaxDiagModels; ++y) gain += covered[c[x]][c[y]] ? 0 : 1;
              if (gain > best_gain) {
                best_gain = gain;
                memcpy(best, c, sizeof(best));
              }
            }
      if (best_gain == 0) break;
      memcpy(subsets[n_pass++], best, sizeof(best));
      for (int x = 0; x < kMaxDiagModels; ++x)
        for (int y = 0; y < kMaxDiagModels; ++y) covered[best[x]][best[y]] = true;
    }
  }
  for (int ps_i = 0; ps_i < n_pass; ++ps_i) {
  const int* sub = subsets[ps_i];
  const bool staged = pl.M > kMaxDiagModels;
  DiagArgs a;
  memset(&a, 0, sizeof(a));
  a.M = pl.m_diag;
  for (int k = 0; k < pl.m_diag; ++k) {
    a.h[k] = p->h[sub[k]];
    a.W[k] = p->W[sub[k]];
    a.d[k] = p->d[sub[k]];
  }
  a.T = p->T;
  a.V = p->V;
  a.labels = p->labels;
  a.ignore_index = p->ignore_index;
  a.n_tt = pl.n_tt_diag;
  a.n_vt = pl.n_vt_diag;
  a.group_v = 4;  // measured: 4 > 8 > 16 here (8 for the forward and backward)
  a.partials = reinterpret_cast<float*>(ws + pl.off_dpart);
  a.rowvals = reinterpret_cast<float*>(ws + pl.off_drow);
  float* sub_out = reinterpret_cast<float*>(ws + pl.off_dsub);
  int32_t* am_sub = reinterpret_cast<int32_t*>(ws + pl.off_dam);
  a.kl_pair = staged ? sub_out : kl_pair;
  a.agree = staged ? sub_out + kMaxDiagModels * kMaxDiagModels : agree;
  a.argmax = staged ? (argmax ? am_sub : nullptr) : argmax;
  hipError_t e;
  {
    ProfScope ps("diag_tiles", s);
    e = launch_diag_tiles(a, pl.f32, pl.wide, s);
  }
  if (e != hipSuccess) return hip_fail(e, "diagnostics tile launch");
  {
    ProfScope ps("diag_reduce", s);
    e = launch_diag_reduce(a, s);
  }
  if (e != hipSuccess) return hip_fail(e, "diagnostics reduction launch");
  if (staged) {
    DiagScatterArgs sc;
    memset(&sc, 0, sizeof(sc));
    sc.M = pl.M;
    sc.n = pl.m_diag;
    for (int k = 0; k < pl.m_diag; ++k) sc.sub[k] = sub[k];
    sc.T = p->T;
    sc.kl_sub = a.kl_pair;
    sc.agree_sub = a.agree;
    sc.am_sub = a.argmax;
    sc.kl_pair = kl_pair;
    sc.agree = agree;
    sc.argmax = argmax;
    {
      ProfScope ps("diag_scatter", s);
      e = launch_diag_scatter(sc, s);
    }
    if (e != hipSuccess) return hip_fail(e, "diagnostics scatter launch");
  }
  }
  return MLS_OK;
}

}  // extern "C"

namespace {

mls_status validate_junction(const mls_junction* j) {
  if (!j) return fail(MLS_INVALID_ARG, "junction is NULL");
  if (j->T < 1 || j->T > (1ll << 31)) return fail(MLS_INVALID_ARG, "T=%lld out of range", (long long)j->T);
  const int64_t wmax = junction_max_width();
  if (j->d_prev < 8 || j->d_fresh < 8 || j->d_prev > wmax || j->d_fresh > wmax)
    return fail(MLS_UNSUPPORTED, "junction widths %lld / %lld outside [8, %lld]", (long long)j->d_prev,
                (long long)j->d_fresh, (long long)wmax);
  if (j->d_prev % 8 || j->d_fresh % 8)
    return fail(MLS_UNSUPPORTED, "junction widths %lld / %lld are not multiples of 8",
                (long long)j->d_prev, (long long)j->d_fresh);
  if ((j->act_dtype != MLS_BF16 && j->act_dtype != MLS_F32) ||
      (j->grad_dtype != MLS_BF16 && j->grad_dtype != MLS_F32))
    return fail(MLS_UNSUPPORTED, "junction dtypes %d / %d unsupported", j->act_dtype, j->grad_dtype);
  if (j->layout != MLS_JUNCTION_PREV_FIRST && j->layout != MLS_JUNCTION_FRESH_FIRST)
    return fail(MLS_INVALID_ARG, "junction layout %d unknown", j->layout);
  if (j->flags & ~(uint32_t)MLS_JUNCTION_ACCUMULATE)
    return fail(MLS_INVALID_ARG, "unknown junction flags 0x%x", j->flags);
  return MLS_OK;
}

bool disjoint(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x + na <= y || y + nb <= x;
}

JunctionArgs junction_args(const mls_junction* j) {
  JunctionArgs a;
  memset(&a, 0, sizeof(a));
  a.T = j->T;
  a.d_prev = j->d_prev;
  a.d_fresh = j->d_fresh;
  a.prev_first = j->layout == MLS_JUNCTION_PREV_FIRST;
  a.accumulate = (j->flags & MLS_JUNCTION_ACCUMULATE) ? 1 : 0;
  return a;
}

}  // namespace

extern "C" {

mls_status mls_junction_fwd(const mls_junction* j, const void* o, const void* e, void* x,
                            void* stream) {
  g_last_error.clear();
  mls_status st = validate_junction(j);
  if (st != MLS_OK) return st;
  if (!o || !e || !x) return fail(MLS_INVALID_ARG, "o, e and x must be non-NULL");
  if (!aligned(o, 16) || !aligned(e, 16) || !aligned(x, 16))
    return fail(MLS_INVALID_ARG, "o, e and x must be 16-byte aligned");
  const size_t es = j->act_dtype == MLS_F32 ? 4 : 2;
  const size_t nx = (size_t)j->T * (j->d_prev + j->d_fresh) * es;
  if (!disjoint(x, nx, o, (size_t)j->T * j->d_prev * es) ||
      !disjoint(x, nx, e, (size_t)j->T * j->d_fresh * es))
    return fail(MLS_INVALID_ARG, "x overlaps o or e");
  JunctionArgs a = junction_args(j);
  a.o = o;
  a.e = e;
  a.x = x;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t err;
  {
    ProfScope ps("junction_fwd", s);
    err = launch_junction_fwd(a, j->act_dtype == MLS_F32, s);
  }
  if (err != hipSuccess) return hip_fail(err, "junction forward launch");
  return MLS_OK;
}

mls_status mls_junction_bwd(const mls_junction* j, const void* o, const void* e, const void* g_x,
                            void* g_o, void* g_e, void* stream) {
  g_last_error.clear();
  mls_status st = validate_junction(j);
  if (st != MLS_OK) return st;
  if (!o || !e || !g_x || !g_o || !g_e)
    return fail(MLS_INVALID_ARG, "o, e, g_x, g_o and g_e must be non-NULL");
  if (!aligned(o, 16) || !aligned(e, 16) || !aligned(g_x, 16) || !aligned(g_o, 16) || !aligned(g_e, 16))
    return fail(MLS_INVALID_ARG, "junction operands must be 16-byte aligned");
  const size_t ea = j->act_dtype == MLS_F32 ? 4 : 2;
  const size_t eg = j->grad_dtype == MLS_F32 ? 4 : 2;
  const size_t T = (size_t)j->T;
  const size_t n_o = T * j->d_prev * ea, n_e = T * j->d_fresh * ea;
  const size_t n_gx = T * (j->d_prev + j->d_fresh) * eg;
  const size_t n_go = T * j->d_prev * eg, n_ge = T * j->d_fresh * eg;
  const void* ins[3] = {o, e, g_x};
  const size_t nin[3] = {n_o, n_e, n_gx};
  for (int i = 0; i < 3; ++i)
    if (!disjoint(g_o, n_go, ins[i], nin[i]) || !disjoint(g_e, n_ge, ins[i], nin[i]))
      return fail(MLS_INVALID_ARG, "g_o / g_e overlap an input");
  if (!disjoint(g_o, n_go, g_e, n_ge)) return fail(MLS_INVALID_ARG, "g_o and g_e overlap");
  JunctionArgs a = junction_args(j);
  a.o = o;
  a.e = e;
  a.g_x = g_x;
  a.g_o = g_o;
  a.g_e = g_e;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t err;
  {
    ProfScope ps("junction_bwd", s);
    err = launch_junction_bwd(a, j->act_dtype == MLS_F32, j->grad_dtype == MLS_F32, s);
  }
  if (err != hipSuccess) return hip_fail(err, "junction backward launch");
  return MLS_OK;
}

}  // extern "C"

namespace {

mls_status validate_sampling(const mls_sampling* s) {
  if (!s) return fail(MLS_INVALID_ARG, "sampling descriptor is NULL");
  if (s->V < 2 || s->V > 65536) return fail(MLS_UNSUPPORTED, "V=%lld outside [2, 65536]", (long long)s->V);
  if (!s->greedy) {
    if (!(s->temperature > 0.f) || !isfinite(s->temperature))
      return fail(MLS_INVALID_ARG, "temperature must be finite and > 0");
    if (!(s->top_p > 0.f) || s->top_p > 1.f) return fail(MLS_INVALID_ARG, "top_p must be in (0, 1]");
  }
  if (s->reserved != 0) return fail(MLS_INVALID_ARG, "reserved field must be 0");
  return MLS_OK;
}

size_t verify_ws_bytes(int64_t batch, int64_t gamma) {
  return align256((size_t)(batch * gamma + batch * (gamma + 1)) * sizeof(RowDist));
}

}  // namespace

extern "C" {

mls_status mls_head_logits(int64_t T, int64_t V, int64_t d, int32_t dtype, const void* o,
                           const void* W, float* logits, void* stream) {
  g_last_error.clear();
  if (T < 1 || T > (1ll << 30) || V < 1 || V > (1ll << 30) || d < 1 || d > (1 << 20))
    return fail(MLS_INVALID_ARG, "T=%lld V=%lld d=%lld out of range", (long long)T, (long long)V,
                (long long)d);
  if (dtype != MLS_BF16 && dtype != MLS_F32) return fail(MLS_UNSUPPORTED, "dtype=%d unsupported", dtype);
  if (d % (dtype == MLS_BF16 ? 8 : 4))
    return fail(MLS_UNSUPPORTED, "d=%lld is not a multiple of %d", (long long)d,
                dtype == MLS_BF16 ? 8 : 4);
  if (!o || !W || !logits) return fail(MLS_INVALID_ARG, "o, W and logits must be non-NULL");
  if (!aligned(o, 16) || !aligned(W, 16) || !aligned(logits, 16))
    return fail(MLS_INVALID_ARG, "o, W and logits must be 16-byte aligned");
  HeadArgs a;
  memset(&a, 0, sizeof(a));
  a.T = T;
  a.V = V;
  a.d = d;
  a.o = o;
  a.W = W;
  a.logits = logits;
  const bool wide = dtype == MLS_BF16 && d % 64 == 0;
  a.n_tt = (int)((T + head_tile() - 1) / head_tile());
  const int rows = wide ? head_tile_rows(true, a.n_tt) : 128;
  a.n_vt = (int)((V + rows - 1) / rows);
  // tile order (groups of vocabulary tiles), measured on the verifier's 714
  // rows with 192-row tiles: groups of 2 or 4 0.731-0.742 ms per decode step,
  // 6 0.756-0.759, 8 0.745-0.750, 16 0.753-0.758, 32 0.79-0.80
  a.group_v = rows == 192 ? 4 : 8;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e;
  {
    ProfScope ps("head_logits", st);
    e = launch_head_logits(a, dtype == MLS_F32, wide, rows, st);
  }
  if (e != hipSuccess) return hip_fail(e, "head logits launch");
  return MLS_OK;
}

static_assert(sizeof(RowDist) == MLS_ROW_PARAMS_BYTES, "row parameter record size");

mls_status mls_sample(const mls_sampling* s, int64_t rows, const float* logits, const float* u,
                      int32_t* tokens, void* params, void* stream) {
  g_last_error.clear();
  mls_status st = validate_sampling(s);
  if (st != MLS_OK) return st;
  if (rows < 1 || rows > (1ll << 31) - 1) return fail(MLS_INVALID_ARG, "rows=%lld out of range", (long long)rows);
  if (!logits || !tokens || (!s->greedy && !u))
    return fail(MLS_INVALID_ARG, "logits, tokens and (unless greedy) u must be non-NULL");
  if (!aligned(logits, 4) || !aligned(u, 4) || !aligned(tokens, 4) || !aligned(params, 4))
    return fail(MLS_INVALID_ARG, "misaligned pointer");
  SampleArgs a;
  memset(&a, 0, sizeof(a));
  a.rows = rows;
  a.V = s->V;
  a.inv_temp = s->greedy ? 1.f : 1.f / s->temperature;
  a.top_p = s->top_p;
  a.greedy = s->greedy ? 1 : 0;
  a.logits = logits;
  a.u = u;
  a.tokens = tokens;
  a.params = s->greedy ? nullptr : static_cast<RowDist*>(params);
  hipStream_t hs = static_cast<hipStream_t>(stream);
  hipError_t e;
  {
    ProfScope ps("sample", hs);
    e = launch_sample(a, row_elems_per_thread(s->V), hs);
  }
  if (e != hipSuccess) return hip_fail(e, "sample launch");
  return MLS_OK;
}

mls_status mls_spec_verify_workspace(int64_t batch, int64_t gamma, size_t* bytes) {
  g_last_error.clear();
  if (batch < 1 || gamma < 0 || batch > (1 << 24) || gamma > 1024)
    return fail(MLS_INVALID_ARG, "batch=%lld gamma=%lld out of range", (long long)batch, (long long)gamma);
  if (!bytes) return fail(MLS_INVALID_ARG, "bytes is NULL");
  *bytes = verify_ws_bytes(batch, gamma);
  return MLS_OK;
}

mls_status mls_spec_verify(const mls_sampling* s, int64_t batch, int64_t gamma,
                           const float* draft_logits, const float* target_logits,
                           const int32_t* draft_tokens, const float* u_accept,
                           const float* u_sample, const void* draft_params,
                           int32_t* n_accepted, int32_t* next_token, void* workspace,
                           size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  mls_status st = validate_sampling(s);
  if (st != MLS_OK) return st;
  if (batch < 1 || gamma < 0 || batch > (1 << 24) || gamma > 1024)
    return fail(MLS_INVALID_ARG, "batch=%lld gamma=%lld out of range", (long long)batch, (long long)gamma);
  if (!target_logits || !n_accepted || !next_token || (gamma > 0 && (!draft_logits || !draft_tokens)))
    return fail(MLS_INVALID_ARG, "logits, draft tokens and outputs must be non-NULL");
  if (!s->greedy && (!u_sample || (gamma > 0 && !u_accept)))
    return fail(MLS_INVALID_ARG, "sampling needs u_accept and u_sample");
  if (!s->greedy && !workspace) return fail(MLS_INVALID_ARG, "sampling needs the workspace");
  if (!s->greedy && workspace_bytes < verify_ws_bytes(batch, gamma))
    return fail(MLS_WORKSPACE_TOO_SMALL, "verification needs %zu workspace bytes, got %zu",
                verify_ws_bytes(batch, gamma), workspace_bytes);
  if (!aligned(workspace, 16) || !aligned(draft_params, 4))
    return fail(MLS_INVALID_ARG, "misaligned workspace or draft_params");
  hipStream_t hs = static_cast<hipStream_t>(stream);
  const int ept = row_elems_per_thread(s->V);
  const float inv_temp = s->greedy ? 1.f : 1.f / s->temperature;
  hipError_t e;
  // workspace: draft rows' records [gamma][batch], then the verifier rows' [batch][gamma + 1]
  RowDist* params = static_cast<RowDist*>(workspace);
  const bool have_draft = draft_params != nullptr && gamma > 0;
  if (!s->greedy) {
    RowParamArgs r;
    memset(&r, 0, sizeof(r));
    r.rows0 = have_draft ? 0 : batch * gamma;
    r.rows1 = batch * (gamma + 1);
    r.V = s->V;
    r.inv_temp = inv_temp;
    r.top_p = s->top_p;
    r.logits0 = draft_logits;
    r.logits1 = target_logits;
    r.params = have_draft ? params + batch * gamma : params;
    {
      ProfScope ps("row_params", hs);
      e = launch_row_params(r, ept, hs);
    }
    if (e != hipSuccess) return hip_fail(e, "row parameter launch");
  }
  VerifyArgs a;
  memset(&a, 0, sizeof(a));
  a.dparams = have_draft ? static_cast<const RowDist*>(draft_params) : params;
  a.tparams = params + batch * gamma;
  a.batch = batch;
  a.V = s->V;
  a.gamma = (int32_t)gamma;
  a.greedy = s->greedy ? 1 : 0;
  a.inv_temp = inv_temp;
  a.top_p = s->top_p;
  a.draft_logits = draft_logits;
  a.target_logits = target_logits;
  a.draft_tokens = draft_tokens;
  a.u_accept = u_accept;
  a.u_sample = u_sample;
  a.n_accepted = n_accepted;
  a.next_token = next_token;
  {
    ProfScope ps("spec_verify", hs);
    e = launch_verify(a, ept, hs);
  }
  if (e != hipSuccess) return hip_fail(e, "verification launch");
  return MLS_OK;
}

mls_status mls_read_stats_header(const mls_problem* p, const void* stats, void* stream,
                                 int32_t* n_valid, int32_t* device_flags) {
  g_last_error.clear();
  mls_status st = validate(p);
  if (st != MLS_OK) return st;
  if (!stats) return fail(MLS_INVALID_ARG, "stats is NULL");
  Plan pl;
  make_plan(p, pl);
  int32_t hdr[2] = {0, 0};
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(hdr, static_cast<const char*>(stats) + pl.header_off, sizeof(hdr),
                                hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync");
  if ((e = hipStreamSynchronize(s)) != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  if (n_valid) *n_valid = hdr[0];
  if (device_flags) *device_flags = hdr[1];
  return MLS_OK;
}

mls_status mls_device_error(const mls_problem* p, const void* stats, void* stream, int32_t* flags) {
  if (!flags) {
    g_last_error.clear();
    return fail(MLS_INVALID_ARG, "flags is NULL");
  }
  return mls_read_stats_header(p, stats, stream, nullptr, flags);
}

mls_status mls_mfma_probe(int32_t random_operands, int32_t iters, float* sink, size_t sink_floats,
                          double* flops, void* stream) {
  g_last_error.clear();
  if (iters < 1 || iters > (1 << 24)) return fail(MLS_INVALID_ARG, "iters=%d out of range", iters);
  if (!flops) return fail(MLS_INVALID_ARG, "flops is NULL");
  *flops = mfma_probe_flops(iters);
  if (!sink) return MLS_OK;  // size query
  if (sink_floats < (size_t)mfma_probe_sink_floats() || !aligned(sink, 4))
    return fail(MLS_INVALID_ARG, "sink needs %lld floats", (long long)mfma_probe_sink_floats());
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  {
    ProfScope ps("mfma_probe", s);
    e = launch_mfma_probe(random_operands ? 1 : 0, iters, sink, s);
  }
  if (e != hipSuccess) return hip_fail(e, "probe launch");
  return MLS_OK;
}

mls_status mls_profile_enable(int32_t enable) {
  g_last_error.clear();
  g_prof.on = enable != 0;
  return MLS_OK;
}

mls_status mls_profile_report(mls_kernel_time* out, int32_t max_entries, int32_t* n_out) {
  g_last_error.clear();
  if (max_entries < 0 || (max_entries > 0 && !out)) return fail(MLS_INVALID_ARG, "bad output array");
  std::vector<mls_kernel_time> rows;
  mls_status st = MLS_OK;
  for (const ProfRec& r : g_prof.recs) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(r.stop);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.start, r.stop);
    if (e != hipSuccess && st == MLS_OK) st = hip_fail(e, "kernel timing");
    size_t k = 0;
    for (; k < rows.size(); ++k)
      if (strncmp(rows[k].name, r.name, sizeof(rows[k].name)) == 0) break;
    if (k == rows.size()) {
      mls_kernel_time t;
      memset(&t, 0, sizeof(t));
      strncpy(t.name, r.name, sizeof(t.name) - 1);
      rows.push_back(t);
    }
    rows[k].launches += 1;
    rows[k].total_ms += ms;
    g_prof.pool.push_back(r.start);
    g_prof.pool.push_back(r.stop);
  }
  g_prof.recs.clear();
  const int32_t n = (int32_t)std::min<size_t>(rows.size(), (size_t)max_entries);
  for (int32_t k = 0; k < n; ++k) out[k] = rows[k];
  if (n_out) *n_out = (int32_t)rows.size();
  return st;
}

}  // extern "C"
