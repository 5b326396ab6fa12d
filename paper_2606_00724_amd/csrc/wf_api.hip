// C ABI of the WaveFilter filter+attend path: argument checks, workspace
// layout and the kernel sequence of every entry point (see wavefilter.h).
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "wf_kernels.hpp"
#include "wf_launch.hpp"

namespace wf {

static thread_local char g_last_error[512] = "";

static wf_status fail(wf_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return s;
}

static wf_status ok() {
  g_last_error[0] = '\0';
  return WF_OK;
}

float effective_scale(const wf_params& p) {
  return p.scale != 0.f ? p.scale : (float)(1.0 / std::sqrt((double)p.head_dim));
}

int device_cu_count() {
  static thread_local int cached_dev = -1, cached_cus = 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (dev != cached_dev) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
            hipSuccess ||
        cus <= 0)
      cus = 256;
    cached_dev = dev;
    cached_cus = cus;
  }
  return cached_cus;
}

// ------------------------------------------------------------ validation

#define WF_TRY_SHAPE(expr)           \
  do {                               \
    wf_status _s = (expr);           \
    if (_s != WF_OK) return _s;      \
  } while (0)

// Fields every entry point uses (not segments, budget).
static wf_status check_shape(const wf_params* p) {
  if (!p) return fail(WF_ERR_INVALID_ARG, "params is NULL");
  if (p->batch < 1 || p->heads < 1)
    return fail(WF_ERR_INVALID_ARG, "batch (%d) and heads (%d) must be >= 1",
                p->batch, p->heads);
  if ((long)p->batch * p->heads > (1L << 24))
    return fail(WF_ERR_UNSUPPORTED, "batch*heads = %ld exceeds 2^24",
                (long)p->batch * p->heads);
  if (p->head_dim != 64 && p->head_dim != 128)
    return fail(WF_ERR_UNSUPPORTED, "head_dim %d: only 64 and 128 are built",
                p->head_dim);
  if (p->q_len < 1) return fail(WF_ERR_INVALID_ARG, "q_len %d < 1", p->q_len);
  if (p->q_len > WF_MAX_Q_LEN)
    return fail(WF_ERR_UNSUPPORTED, "q_len %d exceeds %d", p->q_len,
                (int)WF_MAX_Q_LEN);
  if (p->gen_len < 0) return fail(WF_ERR_INVALID_ARG, "gen_len %d < 0", p->gen_len);
  if (p->levels < 1) return fail(WF_ERR_INVALID_ARG, "levels %d < 1", p->levels);
  if (p->levels > WF_MAX_LEVELS)
    return fail(WF_ERR_UNSUPPORTED, "levels %d exceeds %d", p->levels,
                (int)WF_MAX_LEVELS);
  if (p->ctx_len < (1 << p->levels))
    return fail(WF_ERR_INVALID_ARG, "ctx_len %d is shorter than 2^levels = %d",
                p->ctx_len, 1 << p->levels);
  if (p->ctx_len > (1 << 30))
    return fail(WF_ERR_UNSUPPORTED, "ctx_len %d exceeds 2^30", p->ctx_len);
  if (p->wavelet != WF_HAAR && p->wavelet != WF_DB2)
    return fail(WF_ERR_INVALID_ARG, "unknown wavelet %d", p->wavelet);
  if (p->boundary != WF_EXT_SYMMETRIC && p->boundary != WF_EXT_PERIODIC)
    return fail(WF_ERR_INVALID_ARG, "unknown boundary %d", p->boundary);
  if (p->dtype != WF_BF16 && p->dtype != WF_F32)
    return fail(WF_ERR_INVALID_ARG, "unknown dtype %d", p->dtype);
  if (!std::isfinite(p->scale))
    return fail(WF_ERR_INVALID_ARG, "scale is not finite");
  return WF_OK;
}

static wf_status check_params(const wf_params* p) {
  WF_TRY_SHAPE(check_shape(p));
  const int nJ = p->ctx_len >> p->levels;
  if (p->segments < 1 || p->segments > nJ)
    return fail(WF_ERR_INVALID_ARG, "segments %d outside [1, %d]", p->segments, nJ);
  if (p->budget < 1) return fail(WF_ERR_INVALID_ARG, "budget %d < 1", p->budget);
  if (p->dtype == WF_BF16 && plan_scan(*p).nbuf < 2)
    return fail(WF_ERR_UNSUPPORTED, "query block and pool range do not fit the LDS ring");
  if ((long)p->batch * p->heads *
          (((long)p->budget < ((long)p->segments << p->levels)
                ? (long)p->budget
                : ((long)p->segments << p->levels)) +
           remainder_len(*p) + (long)p->gen_len) > (1L << 31))
    return fail(WF_ERR_UNSUPPORTED, "sparse cache too large");
  return WF_OK;
}

static wf_status check_ptr(const void* ptr, const char* name, bool nullable) {
  if (!ptr) {
    if (nullable) return WF_OK;
    return fail(WF_ERR_INVALID_ARG, "%s is NULL", name);
  }
  if (((uintptr_t)ptr & 15u) != 0)
    return fail(WF_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  return WF_OK;
}

#define WF_TRY(expr)                 \
  do {                               \
    wf_status _s = (expr);           \
    if (_s != WF_OK) return _s;      \
  } while (0)

#define WF_HIP(expr, what)                                                  \
  do {                                                                      \
    hipError_t _e = (expr);                                                 \
    if (_e != hipSuccess)                                                   \
      return fail(WF_ERR_HIP, "%s: %s", what, hipGetErrorString(_e));      \
  } while (0)

// ------------------------------------------------------------ workspace

static size_t up256(size_t x) { return (x + 255) & ~(size_t)255; }

struct Layout {
  size_t logits = 0, sstats = 0, W = 0, seg = 0, cstats = 0,
         wpool = 0, tok = 0, part = 0, pstat = 0, wsum = 0, wpsum = 0, sseg = 0, total = 0;
};

static long keff_of(const wf_params& p) {
  const long pool = (long)p.segments << p.levels;
  return p.budget < pool ? p.budget : pool;
}

// Regions of the workspace, each 256-byte aligned.  The fused entry point on
// the token-level path keeps a log-sum-exp per (block, query) beside each
// coarse logit instead of the scan's per-workgroup statistics (the scan
// forms the pool normalisers from them on chip), and its attention keeps the
// selected tokens on chip.
static Layout layout_for(const wf_params& p, int op, long attn_rows) {
  Layout l;
  const size_t U = (size_t)p.batch * p.heads, B = p.q_len;
  const size_t nJ = (size_t)p.ctx_len >> p.levels;
  const size_t P = (size_t)p.segments << p.levels;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += up256(bytes);
    return at;
  };
  const bool shared = op == WF_OP_SHARED;
  if (shared) op = WF_OP_FUSED;  // the fused regions, then the sums
  const bool fast = op == WF_OP_FUSED && fast_path(p);
  const bool whole = op == WF_OP_FUSED || op == WF_OP_CACHED;  // a whole step
  const bool skim = op == WF_OP_SKIM || whole;
  const bool scan = op == WF_OP_SCAN || whole;
  const bool attn = op == WF_OP_ATTN || whole;
  if (fast) {
    const FastPlan fp = plan_fast(p);
    l.logits = take(U * nJ * 2 * B * sizeof(float));  // block rows: logits, log-sum-exps
    l.sstats = take(U * fp.R * 2 * B * sizeof(float));
  } else if (skim) {
    const SkimPlan sp = plan_skim(p, op == WF_OP_FUSED);  // from A_J otherwise
    l.logits = take(U * B * nJ * sizeof(float));
    l.sstats = take(U * sp.ntiles * 2 * B * sizeof(float));
  }
  if (whole) {
    l.W = take(U * nJ * sizeof(float));
    l.seg = take(U * p.segments * sizeof(int32_t));
  }
  if (scan) {
    // the token-level path forms the pool normalisers inside the scan
    const ScanPlan cp = plan_scan(p);
    if (!fast) l.cstats = take(U * cp.chunks * 2 * B * sizeof(float));
    l.wpool = take(U * P * sizeof(float));
  }
  // a selecting attention keeps its selected tokens on chip
  const bool attn_selects = fast || (op == WF_OP_CACHED && attn_can_select(p, attn_rows));
  if (whole && !attn_selects) l.tok = take(U * keff_of(p) * sizeof(int32_t));
  if (attn) {
    const AttnPlan ap = plan_attn(p, attn_rows);
    l.part = take(U * ap.splits * B * p.head_dim * sizeof(float));
    l.pstat = take(U * ap.splits * 2 * B * sizeof(float));
  }
  if (shared) {
    // W and W' of each sequence, summed over its heads; its shared regions
    const size_t nb = (size_t)p.batch;
    l.wsum = take(nb * nJ * sizeof(float));
    l.wpsum = take(nb * P * sizeof(float));
    l.sseg = take(nb * p.segments * sizeof(int32_t));
  }
  l.total = off;
  return l;
}

static wf_status check_workspace(const void* ws, size_t have, size_t need) {
  if (need == 0) return WF_OK;
  if (!ws) return fail(WF_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (((uintptr_t)ws & 255u) != 0)
    return fail(WF_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  if (have < need)
    return fail(WF_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", have, need);
  return WF_OK;
}

static inline char* at(void* ws, size_t off) { return static_cast<char*>(ws) + off; }

// ------------------------------------------------------------ fused sequence

// Kernel sequences of the fused entry point.  The general path scores the
// coarse coefficients and runs both passes of the token scan; the token-level
// path (bf16, Haar, 3..5 levels, <= 64 query rows) derives the scan's
// normalisers from the skim's block statistics.
static const char* const kGeneralNames[] = {
    "skim_tile", "skim_select", "scan_stats", "scan_weights",
    "scan_select", "sparse_attn", "attn_combine"};
// with bf16 keys, at most 64 query rows and a multiple of 4 coefficients: W
// over all CUs, the top-S in the statistics pass, and when the attention's
// rows allow it the top-k in the attention
static const char* const kGeneralWideNames[] = {
    "skim_tile", "skim_weights", "scan_stats", "scan_weights",
    "scan_select", "sparse_attn", "attn_combine"};
static const char* const kGeneralWideSelectNames[] = {
    "skim_tile", "skim_weights", "scan_stats", "scan_weights", "sparse_attn", "attn_combine"};
static const char* const kFastNames[] = {
    "token_skim", "block_weights", "scan_weights", "sparse_attn", "attn_combine"};
constexpr int kMaxFusedKernels = 7;

static long fused_rows(const wf_params& p) {
  return keff_of(p) + remainder_len(p) + p.gen_len;
}
// the general sequence with its selections in their consumers
static bool general_wide(const wf_params& p) {
  return !fast_path(p) && scan_can_select(p) && ((p.ctx_len >> p.levels) & 3) == 0;
}
static bool general_attn_selects(const wf_params& p) {
  return general_wide(p) && attn_can_select(p, fused_rows(p));
}
static int fused_kernels(const wf_params& p) {
  return fast_path(p) ? 5 : general_attn_selects(p) ? 6 : 7;
}
static const char* const* fused_names(const wf_params& p) {
  if (fast_path(p)) return kFastNames;
  if (general_wide(p)) return general_attn_selects(p) ? kGeneralWideSelectNames : kGeneralWideNames;
  return kGeneralNames;
}

static wf_status fused_impl(const wf_params* p, const void* Q, const void* K,
                            const void* V, const void* Kg, const void* Vg,
                            void* O, int32_t* tok_idx, int32_t* seg_idx,
                            void* ws, size_t ws_bytes, void* stream,
                            void** events, int n_events) {
  WF_TRY(check_params(p));
  WF_TRY(check_ptr(Q, "Q", false));
  WF_TRY(check_ptr(K, "K", false));
  WF_TRY(check_ptr(V, "V", false));
  WF_TRY(check_ptr(O, "O", false));
  WF_TRY(check_ptr(tok_idx, "tok_idx", true));
  WF_TRY(check_ptr(seg_idx, "seg_idx", true));
  if (p->gen_len > 0) {
    WF_TRY(check_ptr(Kg, "Kg", false));
    WF_TRY(check_ptr(Vg, "Vg", false));
  }
  const int nk = fused_kernels(*p);
  const char* const* names = fused_names(*p);
  if (events && n_events < nk + 1)
    return fail(WF_ERR_INVALID_ARG, "n_events %d < %d", n_events, nk + 1);
  const long keff = keff_of(*p);
  const long nrows = keff + remainder_len(*p) + p->gen_len;
  const Layout l = layout_for(*p, WF_OP_FUSED, nrows);
  WF_TRY(check_workspace(ws, ws_bytes, l.total));
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  float* logits = reinterpret_cast<float*>(at(ws, l.logits));
  float* sstats = reinterpret_cast<float*>(at(ws, l.sstats));
  float* W = reinterpret_cast<float*>(at(ws, l.W));
  int32_t* seg = seg_idx ? seg_idx : reinterpret_cast<int32_t*>(at(ws, l.seg));
  float* cstats = reinterpret_cast<float*>(at(ws, l.cstats));
  float* wpool = reinterpret_cast<float*>(at(ws, l.wpool));
  int32_t* tok = tok_idx ? tok_idx : reinterpret_cast<int32_t*>(at(ws, l.tok));
  float* part = reinterpret_cast<float*>(at(ws, l.part));
  float* pstat = reinterpret_cast<float*>(at(ws, l.pstat));
  int k = 0;
  auto mark = [&]() -> hipError_t {
    if (!events) return hipSuccess;
    return hipEventRecord(static_cast<hipEvent_t>(events[k]), s);
  };
  // launch one kernel of the sequence, bracketed by events when timed
  auto step = [&](hipError_t launched) -> wf_status {
    if (launched != hipSuccess)
      return fail(WF_ERR_HIP, "%s: %s", names[k], hipGetErrorString(launched));
    ++k;
    hipError_t e = mark();
    if (e != hipSuccess) return fail(WF_ERR_HIP, "hipEventRecord: %s", hipGetErrorString(e));
    return WF_OK;
  };
  WF_HIP(mark(), "hipEventRecord");
  if (fast_path(*p)) {
    // token logits -> block rows; W of every block; the scan takes the top-S
    // regions and the attention the top-k tokens themselves
    WF_TRY(step(launch_token_skim(*p, Q, K, logits, sstats, s)));
    WF_TRY(step(launch_block_weights(*p, logits, sstats, W, s)));
    WF_TRY(step(launch_scan_select_weights(*p, Q, K, W, logits, seg, wpool, s)));
    WF_TRY(step(launch_attn_select(*p, Q, K, V, wpool, seg, tok_idx, Kg, Vg, nrows, part,
                                   pstat, s)));
  } else {
    const SkimPlan sp = plan_skim(*p, true);
    WF_TRY(step(launch_skim_tiles(*p, true, Q, K, nullptr, logits, sstats, s)));
    if (general_wide(*p)) {
      WF_TRY(step(launch_skim_weights(*p, sp.ntiles, logits, sstats, W, s)));
      WF_TRY(step(launch_scan_select_stats(*p, Q, K, W, seg, cstats, s)));
    } else {
      WF_TRY(step(launch_skim_select(*p, sp.ntiles, logits, sstats, W, seg, s)));
      WF_TRY(step(launch_scan_chunks(*p, 0, Q, K, seg, cstats, wpool, s)));
    }
    WF_TRY(step(launch_scan_chunks(*p, 1, Q, K, seg, cstats, wpool, s)));
    if (general_attn_selects(*p)) {
      WF_TRY(step(launch_attn_select(*p, Q, K, V, wpool, seg, tok_idx, Kg, Vg, nrows, part,
                                     pstat, s)));
    } else {
      WF_TRY(step(launch_scan_select(*p, wpool, seg, tok, s)));
      WF_TRY(step(launch_attn(*p, Q, K, V, tok, (int)keff, Kg, Vg, p->gen_len, nrows,
                              part, pstat, s)));
    }
  }
  WF_TRY(step(launch_attn_combine(*p, nrows, part, pstat, O, s)));
  return ok();
}

// ------------------------------------------------------------ no allocation
//
// wf_filter_attend_noalloc runs the fused sequence on a workspace that the
// library owns: a file-scope device array, one copy per device, present from
// the load of the code object until the process ends.  Host code never
// passes `scratch` itself (in host code the name is a host-side stand-in, not
// a device address); it passes the address hipGetSymbolAddress reports for
// the current device, looked up once per device.
constexpr size_t kScratchBytes = (size_t)WF_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices] = {};

static wf_status scratch_of_current_device(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(WF_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(WF_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(WF_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return WF_OK;
}

static wf_status noalloc_impl(const wf_params* p, const void* Q, const void* K,
                              const void* V, const void* Kg, const void* Vg, void* O,
                              int32_t* tok_idx, int32_t* seg_idx, void* stream) {
  WF_TRY(check_params(p));
  const long nrows = keff_of(*p) + remainder_len(*p) + p->gen_len;
  const size_t need = layout_for(*p, WF_OP_FUSED, nrows).total;
  if (need > kScratchBytes)
    return fail(WF_ERR_WORKSPACE,
                "these parameters need %zu bytes of scratch; the allocation-free entry "
                "point holds %zu (use wf_filter_attend with a workspace)",
                need, kScratchBytes);
  void* ws = nullptr;
  WF_TRY(scratch_of_current_device(&ws));
  return fused_impl(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx, ws, kScratchBytes, stream,
                    nullptr, 0);
}

// ------------------------------------------------------------ cached A_J

static const char* const kCachedNames[] = {
    "skim_tile", "skim_select", "scan_stats", "scan_weights",
    "scan_select", "sparse_attn", "attn_combine"};
constexpr int kCachedKernels = 7;
// with bf16 keys the attention takes the top-k of W' itself
static const char* const kCachedSelectNames[] = {
    "skim_tile", "skim_select", "scan_stats", "scan_weights", "sparse_attn", "attn_combine"};
// with bf16 keys and at most 64 query rows W is formed over all CUs and the
// statistics pass takes the top-S of W itself
static const char* const kCachedWideNames[] = {
    "skim_tile", "skim_weights", "scan_stats", "scan_weights",
    "scan_select", "sparse_attn", "attn_combine"};
static const char* const kCachedWideSelectNames[] = {
    "skim_tile", "skim_weights", "scan_stats", "scan_weights", "sparse_attn", "attn_combine"};

static long cached_rows(const wf_params& p) {
  return keff_of(p) + remainder_len(p) + p.gen_len;
}
static bool cached_attn_selects(const wf_params& p) {
  return attn_can_select(p, cached_rows(p));
}
static bool cached_scan_selects(const wf_params& p) {
  return scan_can_select(p) && ((p.ctx_len >> p.levels) & 3) == 0;
}
static int cached_kernels(const wf_params& p) {
  return cached_attn_selects(p) ? kCachedKernels - 1 : kCachedKernels;
}
static const char* const* cached_names(const wf_params& p) {
  if (cached_scan_selects(p))
    return cached_attn_selects(p) ? kCachedWideSelectNames : kCachedWideNames;
  return cached_attn_selects(p) ? kCachedSelectNames : kCachedNames;
}

static wf_status cached_impl(const wf_params* p, const void* Q, const float* approx,
                             const void* K, const void* V, const void* Kg, const void* Vg,
                             void* O, int32_t* tok_idx, int32_t* seg_idx, void* ws,
                             size_t ws_bytes, void* stream, void** events, int n_events) {
  WF_TRY(check_params(p));
  WF_TRY(check_ptr(Q, "Q", false));
  WF_TRY(check_ptr(approx, "approx", false));
  WF_TRY(check_ptr(K, "K", false));
  WF_TRY(check_ptr(V, "V", false));
  WF_TRY(check_ptr(O, "O", false));
  WF_TRY(check_ptr(tok_idx, "tok_idx", true));
  WF_TRY(check_ptr(seg_idx, "seg_idx", true));
  if (p->gen_len > 0) {
    WF_TRY(check_ptr(Kg, "Kg", false));
    WF_TRY(check_ptr(Vg, "Vg", false));
  }
  const int nk = cached_kernels(*p);
  const char* const* names = cached_names(*p);
  if (events && n_events < nk + 1)
    return fail(WF_ERR_INVALID_ARG, "n_events %d < %d", n_events, nk + 1);
  const long keff = keff_of(*p);
  const long nrows = cached_rows(*p);
  const Layout l = layout_for(*p, WF_OP_CACHED, nrows);
  WF_TRY(check_workspace(ws, ws_bytes, l.total));
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  float* logits = reinterpret_cast<float*>(at(ws, l.logits));
  float* sstats = reinterpret_cast<float*>(at(ws, l.sstats));
  float* W = reinterpret_cast<float*>(at(ws, l.W));
  int32_t* seg = seg_idx ? seg_idx : reinterpret_cast<int32_t*>(at(ws, l.seg));
  float* cstats = reinterpret_cast<float*>(at(ws, l.cstats));
  float* wpool = reinterpret_cast<float*>(at(ws, l.wpool));
  int32_t* tok = tok_idx ? tok_idx : reinterpret_cast<int32_t*>(at(ws, l.tok));
  float* part = reinterpret_cast<float*>(at(ws, l.part));
  float* pstat = reinterpret_cast<float*>(at(ws, l.pstat));
  int k = 0;
  auto mark = [&]() -> hipError_t {
    if (!events) return hipSuccess;
    return hipEventRecord(static_cast<hipEvent_t>(events[k]), s);
  };
  auto step = [&](hipError_t launched) -> wf_status {
    if (launched != hipSuccess)
      return fail(WF_ERR_HIP, "%s: %s", names[k], hipGetErrorString(launched));
    ++k;
    hipError_t e = mark();
    if (e != hipSuccess) return fail(WF_ERR_HIP, "hipEventRecord: %s", hipGetErrorString(e));
    return WF_OK;
  };
  WF_HIP(mark(), "hipEventRecord");
  const SkimPlan sp = plan_skim(*p, false);
  WF_TRY(step(launch_skim_tiles(*p, false, Q, nullptr, approx, logits, sstats, s)));
  if (cached_scan_selects(*p)) {
    WF_TRY(step(launch_skim_weights(*p, sp.ntiles, logits, sstats, W, s)));
    WF_TRY(step(launch_scan_select_stats(*p, Q, K, W, seg, cstats, s)));
  } else {
    WF_TRY(step(launch_skim_select(*p, sp.ntiles, logits, sstats, W, seg, s)));
    WF_TRY(step(launch_scan_chunks(*p, 0, Q, K, seg, cstats, wpool, s)));
  }
  WF_TRY(step(launch_scan_chunks(*p, 1, Q, K, seg, cstats, wpool, s)));
  if (cached_attn_selects(*p)) {
    WF_TRY(step(launch_attn_select(*p, Q, K, V, wpool, seg, tok_idx, Kg, Vg, nrows, part,
                                   pstat, s)));
  } else {
    WF_TRY(step(launch_scan_select(*p, wpool, seg, tok, s)));
    WF_TRY(step(launch_attn(*p, Q, K, V, tok, (int)keff, Kg, Vg, p->gen_len, nrows, part,
                            pstat, s)));
  }
  WF_TRY(step(launch_attn_combine(*p, nrows, part, pstat, O, s)));
  return ok();
}

// ------------------------------------------------------------ shared selection

// One selection per sequence, shared by its heads: the token-level sequence
// with W and W' added over the heads before each top-k.
static const char* const kSharedNames[] = {
    "token_skim", "block_weights", "head_sum_w", "scan_weights",
    "head_sum_wpool", "sparse_attn", "attn_combine"};
// the general path: W per unit from the skim select (whose own regions are
// not used), the heads' sum, one select per sequence; the scan's two passes
// per unit over the sequence's regions, the heads' sum of W', one token
// select per sequence; attention per unit
static const char* const kSharedGeneralNames[] = {
    "skim_tile", "skim_select", "head_sum_w", "select_regions", "scan_stats",
    "scan_weights", "head_sum_wpool", "scan_select", "sparse_attn", "attn_combine"};
// with a multiple of 4 coefficients each head's W alone, over all CUs
static const char* const kSharedGeneralWideNames[] = {
    "skim_tile", "skim_weights", "head_sum_w", "select_regions", "scan_stats",
    "scan_weights", "head_sum_wpool", "scan_select", "sparse_attn", "attn_combine"};
constexpr int kSharedMaxKernels = 10;
static bool shared_w_only(const wf_params& p) { return ((p.ctx_len >> p.levels) & 3) == 0; }
static int shared_kernels(const wf_params& p) { return fast_path(p) ? 7 : 10; }
static const char* const* shared_names(const wf_params& p) {
  if (fast_path(p)) return kSharedNames;
  return shared_w_only(p) ? kSharedGeneralWideNames : kSharedGeneralNames;
}

static wf_status shared_impl(const wf_params* p, const void* Q, const void* K,
                             const void* V, const void* Kg, const void* Vg, void* O,
                             int32_t* tok_idx, int32_t* seg_idx, void* ws, size_t ws_bytes,
                             void* stream, void** events, int n_events) {
  WF_TRY(check_params(p));
  WF_TRY(check_ptr(Q, "Q", false));
  WF_TRY(check_ptr(K, "K", false));
  WF_TRY(check_ptr(V, "V", false));
  WF_TRY(check_ptr(O, "O", false));
  WF_TRY(check_ptr(tok_idx, "tok_idx", true));
  WF_TRY(check_ptr(seg_idx, "seg_idx", true));
  if (p->gen_len > 0) {
    WF_TRY(check_ptr(Kg, "Kg", false));
    WF_TRY(check_ptr(Vg, "Vg", false));
  }
  const int nk = shared_kernels(*p);
  const char* const* names = shared_names(*p);
  if (events && n_events < nk + 1)
    return fail(WF_ERR_INVALID_ARG, "n_events %d < %d", n_events, nk + 1);
  const long keff = keff_of(*p);
  const long nrows = keff + remainder_len(*p) + p->gen_len;
  const Layout l = layout_for(*p, WF_OP_SHARED, nrows);
  WF_TRY(check_workspace(ws, ws_bytes, l.total));
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  float* logits = reinterpret_cast<float*>(at(ws, l.logits));
  float* sstats = reinterpret_cast<float*>(at(ws, l.sstats));
  float* W = reinterpret_cast<float*>(at(ws, l.W));
  float* cstats = reinterpret_cast<float*>(at(ws, l.cstats));
  float* wpool = reinterpret_cast<float*>(at(ws, l.wpool));
  float* part = reinterpret_cast<float*>(at(ws, l.part));
  float* pstat = reinterpret_cast<float*>(at(ws, l.pstat));
  float* wsum = reinterpret_cast<float*>(at(ws, l.wsum));
  float* wpsum = reinterpret_cast<float*>(at(ws, l.wpsum));
  int32_t* seg = seg_idx ? seg_idx : reinterpret_cast<int32_t*>(at(ws, l.sseg));
  const int H = p->heads;
  const long nJ = (long)p->ctx_len >> p->levels;
  const long P = (long)p->segments << p->levels;
  int k = 0;
  auto mark = [&]() -> hipError_t {
    if (!events) return hipSuccess;
    return hipEventRecord(static_cast<hipEvent_t>(events[k]), s);
  };
  auto step = [&](hipError_t launched) -> wf_status {
    if (launched != hipSuccess)
      return fail(WF_ERR_HIP, "%s: %s", names[k], hipGetErrorString(launched));
    ++k;
    hipError_t e = mark();
    if (e != hipSuccess) return fail(WF_ERR_HIP, "hipEventRecord: %s", hipGetErrorString(e));
    return WF_OK;
  };
  WF_HIP(mark(), "hipEventRecord");
  if (fast_path(*p)) {
    WF_TRY(step(launch_token_skim(*p, Q, K, logits, sstats, s)));
    WF_TRY(step(launch_block_weights(*p, logits, sstats, W, s)));
    WF_TRY(step(launch_head_sum(W, wsum, nJ, H, p->batch, s)));
    WF_TRY(step(launch_scan_select_weights(*p, Q, K, wsum, logits, seg, wpool, s, H)));
    WF_TRY(step(launch_head_sum(wpool, wpsum, P, H, p->batch, s)));
    WF_TRY(step(launch_attn_select(*p, Q, K, V, wpsum, seg, tok_idx, Kg, Vg, nrows, part,
                                   pstat, s, H)));
  } else {
    // one "unit" per sequence for the two selections over the heads' sums
    wf_params pg = *p;
    pg.heads = 1;
    int32_t* unit_seg = reinterpret_cast<int32_t*>(at(ws, l.seg));  // not used after
    int32_t* tok = tok_idx ? tok_idx : reinterpret_cast<int32_t*>(at(ws, l.tok));
    const SkimPlan sp = plan_skim(*p, true);
    WF_TRY(step(launch_skim_tiles(*p, true, Q, K, nullptr, logits, sstats, s)));
    if (shared_w_only(*p))
      WF_TRY(step(launch_skim_weights(*p, sp.ntiles, logits, sstats, W, s)));
    else  // the per-unit select's regions are not used
      WF_TRY(step(launch_skim_select(*p, sp.ntiles, logits, sstats, W, unit_seg, s)));
    WF_TRY(step(launch_head_sum(W, wsum, nJ, H, p->batch, s)));
    WF_TRY(step(launch_select_w(pg, p->batch, wsum, seg, s)));
    WF_TRY(step(launch_scan_chunks(*p, 0, Q, K, seg, cstats, wpool, s, 0, H)));
    WF_TRY(step(launch_scan_chunks(*p, 1, Q, K, seg, cstats, wpool, s, 0, H)));
    WF_TRY(step(launch_head_sum(wpool, wpsum, P, H, p->batch, s)));
    WF_TRY(step(launch_scan_select(pg, wpsum, seg, tok, s)));
    WF_TRY(step(launch_attn(*p, Q, K, V, tok, (int)keff, Kg, Vg, p->gen_len, nrows, part,
                            pstat, s, H)));
  }
  WF_TRY(step(launch_attn_combine(*p, nrows, part, pstat, O, s)));
  return ok();
}

// ------------------------------------------------------------ recursion

// Validates the recursion's parameters and fills counts[b - 1] = c_b.
static wf_status check_recursion(const wf_params* p, const float* prop, int32_t* counts) {
  WF_TRY(check_shape(p));
  if (!prop) return fail(WF_ERR_INVALID_ARG, "proportions is NULL");
  long n = (long)p->ctx_len >> p->levels;
  for (int b = p->levels; b >= 1; --b) {
    const float m = prop[b - 1];
    if (!(m > 0.f && m <= 1.f))
      return fail(WF_ERR_INVALID_ARG, "proportion m_%d = %g outside (0, 1]", b, (double)m);
    long c = (long)std::ceil((double)m * (double)n);
    c = std::max(1L, std::min(c, n));
    counts[b - 1] = (int32_t)c;
    n = 2 * c;
  }
  if ((long)p->batch * p->heads * (2L * counts[0] + remainder_len(*p) + p->gen_len) >
      (1L << 31))
    return fail(WF_ERR_UNSUPPORTED, "sparse cache too large");
  return WF_OK;
}

struct RecLayout {
  size_t logits = 0, stats = 0, W = 0, sel[2] = {0, 0}, tok = 0, part = 0, pstat = 0,
         total = 0;
};

static RecLayout rec_layout(const wf_params& p, const int32_t* counts) {
  RecLayout l;
  const RecPlan rp = plan_recursion(p, counts);
  const size_t U = (size_t)p.batch * p.heads, B = p.q_len;
  const long nrows = 2L * counts[0] + remainder_len(p) + p.gen_len;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += up256(bytes);
    return at;
  };
  l.logits = take(U * B * rp.max_n * sizeof(float));
  l.stats = take(U * rp.max_tiles * 2 * B * sizeof(float));
  l.W = take(U * rp.max_n * sizeof(float));
  l.sel[0] = take(U * rp.max_keep * sizeof(int32_t));
  l.sel[1] = take(U * rp.max_keep * sizeof(int32_t));
  l.tok = take(U * 2 * counts[0] * sizeof(int32_t));
  const AttnPlan ap = plan_attn(p, nrows);
  l.part = take(U * ap.splits * B * p.head_dim * sizeof(float));
  l.pstat = take(U * ap.splits * 2 * B * sizeof(float));
  l.total = off;
  return l;
}

static const char* const kRecTileNames[WF_MAX_LEVELS] = {
    "rec_tiles_b1", "rec_tiles_b2", "rec_tiles_b3", "rec_tiles_b4", "rec_tiles_b5",
    "rec_tiles_b6", "rec_tiles_b7", "rec_tiles_b8", "rec_tiles_b9", "rec_tiles_b10"};
static const char* const kRecSelectNames[WF_MAX_LEVELS] = {
    "rec_select_b1", "rec_select_b2", "rec_select_b3", "rec_select_b4", "rec_select_b5",
    "rec_select_b6", "rec_select_b7", "rec_select_b8", "rec_select_b9", "rec_select_b10"};

static int rec_kernels(const wf_params& p) { return 2 * p.levels + 2; }

static const char* rec_kernel_name(const wf_params& p, int i) {
  if (i < 2 * p.levels) {
    const int b = p.levels - i / 2;
    return (i % 2 == 0 ? kRecTileNames : kRecSelectNames)[b - 1];
  }
  return i == 2 * p.levels ? "sparse_attn" : "attn_combine";
}

static wf_status recursive_impl(const wf_params* p, const float* prop, const void* Q,
                                const void* K, const void* V, const void* Kg,
                                const void* Vg, void* O, int32_t* tok_idx,
                                int32_t* kept_idx, void* ws, size_t ws_bytes,
                                void* stream, void** events, int n_events) {
  int32_t counts[WF_MAX_LEVELS];
  WF_TRY(check_recursion(p, prop, counts));
  WF_TRY(check_ptr(Q, "Q", false));
  WF_TRY(check_ptr(K, "K", false));
  WF_TRY(check_ptr(V, "V", false));
  WF_TRY(check_ptr(O, "O", false));
  WF_TRY(check_ptr(tok_idx, "tok_idx", true));
  if (kept_idx && ((uintptr_t)kept_idx & 3u) != 0)
    return fail(WF_ERR_INVALID_ARG, "kept_idx is not 4-byte aligned");
  if (p->gen_len > 0) {
    WF_TRY(check_ptr(Kg, "Kg", false));
    WF_TRY(check_ptr(Vg, "Vg", false));
  }
  const int nk = rec_kernels(*p);
  if (events && n_events < nk + 1)
    return fail(WF_ERR_INVALID_ARG, "n_events %d < %d", n_events, nk + 1);
  const RecLayout l = rec_layout(*p, counts);
  WF_TRY(check_workspace(ws, ws_bytes, l.total));
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  float* logits = reinterpret_cast<float*>(at(ws, l.logits));
  float* stats = reinterpret_cast<float*>(at(ws, l.stats));
  float* W = reinterpret_cast<float*>(at(ws, l.W));
  int32_t* sel[2] = {reinterpret_cast<int32_t*>(at(ws, l.sel[0])),
                     reinterpret_cast<int32_t*>(at(ws, l.sel[1]))};
  int32_t* tok = tok_idx ? tok_idx : reinterpret_cast<int32_t*>(at(ws, l.tok));
  float* part = reinterpret_cast<float*>(at(ws, l.part));
  float* pstat = reinterpret_cast<float*>(at(ws, l.pstat));
  int k = 0;
  auto mark = [&]() -> hipError_t {
    if (!events) return hipSuccess;
    return hipEventRecord(static_cast<hipEvent_t>(events[k]), s);
  };
  auto step = [&](hipError_t launched) -> wf_status {
    if (launched != hipSuccess)
      return fail(WF_ERR_HIP, "%s: %s", rec_kernel_name(*p, k), hipGetErrorString(launched));
    ++k;
    hipError_t e = mark();
    if (e != hipSuccess) return fail(WF_ERR_HIP, "hipEventRecord: %s", hipGetErrorString(e));
    return WF_OK;
  };
  WF_HIP(mark(), "hipEventRecord");
  long n = (long)p->ctx_len >> p->levels;
  const int32_t* parent = nullptr;
  int npar = 0;
  const long U = (long)p->batch * p->heads;
  long kept_at = 0;  // element offset of this scale's ids in kept_idx
  for (int b = p->levels; b >= 1; --b) {
    int32_t* out = b == 1 ? tok : kept_idx ? kept_idx + kept_at : sel[b & 1];
    kept_at += U * counts[b - 1];
    if (rec_token_path(*p) && b <= 5) {
      // the scale's coarse logits as sums of token logits (of the kept
      // blocks' tokens below the first scale)
      const long rows = parent ? (long)npar << (b + 1) : filtered_len(*p);
      WF_TRY(step(launch_rec_token_skim(*p, b, n, parent, npar, Q, K, logits, stats, s)));
      WF_TRY(step(launch_rec_select_slices(*p, b, n, counts[b - 1], parent, npar,
                                           plan_rec_token(*p, b, rows, parent != nullptr).R,
                                           logits, stats, W, out, s)));
    } else {
      WF_TRY(step(launch_rec_tiles(*p, b, n, parent, npar, Q, K, logits, stats, s)));
      WF_TRY(step(launch_rec_select(*p, b, n, counts[b - 1], parent, npar, logits, stats, W,
                                    out, s)));
    }
    parent = out;
    npar = counts[b - 1];
    n = 2L * counts[b - 1];
  }
  const int nsel = 2 * counts[0];
  const long nrows = (long)nsel + remainder_len(*p) + p->gen_len;
  WF_TRY(step(launch_attn(*p, Q, K, V, tok, nsel, Kg, Vg, p->gen_len, nrows, part, pstat,
                          s)));
  WF_TRY(step(launch_attn_combine(*p, nrows, part, pstat, O, s)));
  return ok();
}

}  // namespace wf

using namespace wf;

extern "C" {

size_t wf_workspace_bytes(const wf_params* p, int32_t op) {
  if (check_params(p) != WF_OK) return 0;
  if (op < WF_OP_SKIM || op > WF_OP_SHARED) return 0;
  return layout_for(*p, op, keff_of(*p) + remainder_len(*p) + p->gen_len).total;
}

int32_t wf_effective_budget(const wf_params* p) {
  if (check_params(p) != WF_OK) return -1;
  return (int32_t)keff_of(*p);
}

wf_status wf_dwt_keys(const wf_params* p, const void* K, float* approx,
                      float* details, void* stream) {
  WF_TRY(check_params(p));
  WF_TRY(check_ptr(K, "K", false));
  WF_TRY(check_ptr(approx, "approx", false));
  WF_TRY(check_ptr(details, "details", true));
  (void)hipGetLastError();
  WF_HIP(launch_dwt(*p, K, approx, details, static_cast<hipStream_t>(stream)),
         "dwt");
  return ok();
}

wf_status wf_skim_score(const wf_params* p, const void* Q, const float* approx,
                        float* seg_score, int32_t* seg_idx, void* workspace,
                        size_t workspace_bytes, void* stream) {
  WF_TRY(check_params(p));
  WF_TRY(check_ptr(Q, "Q", false));
  WF_TRY(check_ptr(approx, "approx", false));
  WF_TRY(check_ptr(seg_score, "seg_score", false));
  WF_TRY(check_ptr(seg_idx, "seg_idx", false));
  const Layout l = layout_for(*p, WF_OP_SKIM, 0);
  WF_TRY(check_workspace(workspace, workspace_bytes, l.total));
  hipStream_t s = static_cast<hipStream_t>(stream);
  const SkimPlan sp = plan_skim(*p, false);
  float* logits = reinterpret_cast<float*>(at(workspace, l.logits));
  float* sstats = reinterpret_cast<float*>(at(workspace, l.sstats));
  (void)hipGetLastError();
  WF_HIP(launch_skim_tiles(*p, false, Q, nullptr, approx, logits, sstats, s),
         "skim_tile");
  WF_HIP(launch_skim_select(*p, sp.ntiles, logits, sstats, seg_score, seg_idx, s),
         "skim_select");
  return ok();
}

wf_status wf_scan_select(const wf_params* p, const void* Q, const void* K,
                         const int32_t* seg_idx, float* tok_score,
                         int32_t* tok_idx, void* workspace,
                         size_t workspace_bytes, void* stream) {
  WF_TRY(check_params(p));
  WF_TRY(check_ptr(Q, "Q", false));
  WF_TRY(check_ptr(K, "K", false));
  WF_TRY(check_ptr(seg_idx, "seg_idx", false));
  WF_TRY(check_ptr(tok_score, "tok_score", true));
  WF_TRY(check_ptr(tok_idx, "tok_idx", false));
  const Layout l = layout_for(*p, WF_OP_SCAN, 0);
  WF_TRY(check_workspace(workspace, workspace_bytes, l.total));
  hipStream_t s = static_cast<hipStream_t>(stream);
  float* cstats = reinterpret_cast<float*>(at(workspace, l.cstats));
  float* wpool = tok_score ? tok_score : reinterpret_cast<float*>(at(workspace, l.wpool));
  (void)hipGetLastError();
  WF_HIP(launch_scan_chunks(*p, 0, Q, K, seg_idx, cstats, wpool, s), "scan_stats");
  WF_HIP(launch_scan_chunks(*p, 1, Q, K, seg_idx, cstats, wpool, s), "scan_weights");
  WF_HIP(launch_scan_select(*p, wpool, seg_idx, tok_idx, s), "scan_select");
  return ok();
}

wf_status wf_gather_kv(const wf_params* p, const void* K, const void* V,
                       const int32_t* tok_idx, const void* Kg, const void* Vg,
                       void* Ks, void* Vs, void* stream) {
  WF_TRY(check_params(p));
  WF_TRY(check_ptr(K, "K", false));
  WF_TRY(check_ptr(V, "V", false));
  WF_TRY(check_ptr(tok_idx, "tok_idx", false));
  WF_TRY(check_ptr(Ks, "Ks", false));
  WF_TRY(check_ptr(Vs, "Vs", false));
  if (p->gen_len > 0) {
    WF_TRY(check_ptr(Kg, "Kg", false));
    WF_TRY(check_ptr(Vg, "Vg", false));
  }
  (void)hipGetLastError();
  WF_HIP(launch_gather(*p, K, V, tok_idx, Kg, Vg, Ks, Vs,
                       static_cast<hipStream_t>(stream)),
         "gather");
  return ok();
}

wf_status wf_sparse_attn(const wf_params* p, const void* Q, const void* Ks,
                         const void* Vs, int32_t n_kv, void* O,
                         void* workspace, size_t workspace_bytes,
                         void* stream) {
  WF_TRY(check_params(p));
  WF_TRY(check_ptr(Q, "Q", false));
  WF_TRY(check_ptr(Ks, "Ks", false));
  WF_TRY(check_ptr(Vs, "Vs", false));
  WF_TRY(check_ptr(O, "O", false));
  if (n_kv < 1) return fail(WF_ERR_INVALID_ARG, "n_kv %d < 1", n_kv);
  const Layout l = layout_for(*p, WF_OP_ATTN, n_kv);
  WF_TRY(check_workspace(workspace, workspace_bytes, l.total));
  hipStream_t s = static_cast<hipStream_t>(stream);
  float* part = reinterpret_cast<float*>(at(workspace, l.part));
  float* pstat = reinterpret_cast<float*>(at(workspace, l.pstat));
  (void)hipGetLastError();
  WF_HIP(launch_attn(*p, Q, Ks, Vs, nullptr, n_kv, nullptr, nullptr, 0, n_kv,
                     part, pstat, s),
         "sparse_attn");
  WF_HIP(launch_attn_combine(*p, n_kv, part, pstat, O, s), "attn_combine");
  return ok();
}

wf_status wf_filter_attend(const wf_params* p, const void* Q, const void* K,
                           const void* V, const void* Kg, const void* Vg,
                           void* O, int32_t* tok_idx, int32_t* seg_idx,
                           void* workspace, size_t workspace_bytes,
                           void* stream) {
  return fused_impl(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx, workspace,
                    workspace_bytes, stream, nullptr, 0);
}

wf_status wf_filter_attend_timed(const wf_params* p, const void* Q,
                                 const void* K, const void* V, const void* Kg,
                                 const void* Vg, void* O, int32_t* tok_idx,
                                 int32_t* seg_idx, void* workspace,
                                 size_t workspace_bytes, void* stream,
                                 void** events, int32_t n_events) {
  if (!events) return fail(WF_ERR_INVALID_ARG, "events is NULL");
  for (int i = 0; i < n_events && i <= kMaxFusedKernels; ++i)
    if (!events[i]) return fail(WF_ERR_INVALID_ARG, "events[%d] is NULL", i);
  return fused_impl(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx, workspace,
                    workspace_bytes, stream, events, n_events);
}

wf_status wf_filter_attend_noalloc(const wf_params* p, const void* Q, const void* K,
                                   const void* V, const void* Kg, const void* Vg, void* O,
                                   int32_t* tok_idx, int32_t* seg_idx, void* stream) {
  return noalloc_impl(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx, stream);
}

int32_t wf_filter_attend_kernels(const wf_params* p) {
  if (check_params(p) != WF_OK) return -1;
  return fused_kernels(*p);
}

const char* wf_filter_attend_kernel_name(const wf_params* p, int32_t i) {
  if (check_params(p) != WF_OK || i < 0 || i >= fused_kernels(*p)) return nullptr;
  return fused_names(*p)[i];
}

wf_status wf_filter_attend_shared(const wf_params* p, const void* Q, const void* K,
                                  const void* V, const void* Kg, const void* Vg, void* O,
                                  int32_t* tok_idx, int32_t* seg_idx, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  return shared_impl(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx, workspace, workspace_bytes,
                     stream, nullptr, 0);
}

wf_status wf_filter_attend_shared_timed(const wf_params* p, const void* Q, const void* K,
                                        const void* V, const void* Kg, const void* Vg,
                                        void* O, int32_t* tok_idx, int32_t* seg_idx,
                                        void* workspace, size_t workspace_bytes,
                                        void* stream, void** events, int32_t n_events) {
  if (!events) return fail(WF_ERR_INVALID_ARG, "events is NULL");
  for (int i = 0; i < n_events && i <= kSharedMaxKernels; ++i)
    if (!events[i]) return fail(WF_ERR_INVALID_ARG, "events[%d] is NULL", i);
  return shared_impl(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx, workspace, workspace_bytes,
                     stream, events, n_events);
}

int32_t wf_filter_attend_shared_kernels(const wf_params* p) {
  if (check_params(p) != WF_OK) return -1;
  return shared_kernels(*p);
}

const char* wf_filter_attend_shared_kernel_name(const wf_params* p, int32_t i) {
  if (check_params(p) != WF_OK || i < 0 || i >= shared_kernels(*p)) return nullptr;
  return shared_names(*p)[i];
}

wf_status wf_filter_attend_cached(const wf_params* p, const void* Q, const float* approx,
                                  const void* K, const void* V, const void* Kg,
                                  const void* Vg, void* O, int32_t* tok_idx,
                                  int32_t* seg_idx, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  return cached_impl(p, Q, approx, K, V, Kg, Vg, O, tok_idx, seg_idx, workspace,
                     workspace_bytes, stream, nullptr, 0);
}

wf_status wf_filter_attend_cached_timed(const wf_params* p, const void* Q,
                                        const float* approx, const void* K, const void* V,
                                        const void* Kg, const void* Vg, void* O,
                                        int32_t* tok_idx, int32_t* seg_idx, void* workspace,
                                        size_t workspace_bytes, void* stream, void** events,
                                        int32_t n_events) {
  if (!events) return fail(WF_ERR_INVALID_ARG, "events is NULL");
  for (int i = 0; i < n_events && i <= cached_kernels(*p); ++i)
    if (!events[i]) return fail(WF_ERR_INVALID_ARG, "events[%d] is NULL", i);
  return cached_impl(p, Q, approx, K, V, Kg, Vg, O, tok_idx, seg_idx, workspace,
                     workspace_bytes, stream, events, n_events);
}

int32_t wf_filter_attend_cached_kernels(const wf_params* p) {
  if (check_params(p) != WF_OK) return -1;
  return cached_kernels(*p);
}

const char* wf_filter_attend_cached_kernel_name(const wf_params* p, int32_t i) {
  if (check_params(p) != WF_OK || i < 0 || i >= cached_kernels(*p)) return nullptr;
  return cached_names(*p)[i];
}

wf_status wf_recursion_counts(const wf_params* p, const float* proportions,
                              int32_t* counts) {
  int32_t c[WF_MAX_LEVELS];
  if (!counts) return fail(WF_ERR_INVALID_ARG, "counts is NULL");
  WF_TRY(check_recursion(p, proportions, c));
  for (int b = 0; b < p->levels; ++b) counts[b] = c[b];
  return ok();
}

size_t wf_recursive_workspace_bytes(const wf_params* p, const float* proportions) {
  int32_t c[WF_MAX_LEVELS];
  if (check_recursion(p, proportions, c) != WF_OK) return 0;
  return rec_layout(*p, c).total;
}

wf_status wf_filter_attend_recursive(const wf_params* p, const float* proportions,
                                     const void* Q, const void* K, const void* V,
                                     const void* Kg, const void* Vg, void* O,
                                     int32_t* tok_idx, int32_t* kept_idx, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  return recursive_impl(p, proportions, Q, K, V, Kg, Vg, O, tok_idx, kept_idx, workspace,
                        workspace_bytes, stream, nullptr, 0);
}

wf_status wf_filter_attend_recursive_timed(const wf_params* p, const float* proportions,
                                           const void* Q, const void* K, const void* V,
                                           const void* Kg, const void* Vg, void* O,
                                           int32_t* tok_idx, int32_t* kept_idx,
                                           void* workspace, size_t workspace_bytes,
                                           void* stream, void** events, int32_t n_events) {
  if (!events) return fail(WF_ERR_INVALID_ARG, "events is NULL");
  WF_TRY(check_shape(p));
  for (int i = 0; i < n_events && i <= rec_kernels(*p); ++i)
    if (!events[i]) return fail(WF_ERR_INVALID_ARG, "events[%d] is NULL", i);
  return recursive_impl(p, proportions, Q, K, V, Kg, Vg, O, tok_idx, kept_idx, workspace,
                        workspace_bytes, stream, events, n_events);
}

int32_t wf_filter_attend_recursive_kernels(const wf_params* p) {
  if (check_shape(p) != WF_OK) return -1;
  return rec_kernels(*p);
}

const char* wf_filter_attend_recursive_kernel_name(const wf_params* p, int32_t i) {
  if (check_shape(p) != WF_OK || i < 0 || i >= rec_kernels(*p)) return nullptr;
  return rec_kernel_name(*p, i);
}

wf_status wf_init(void) {
  WF_HIP(load_fast_kernels(), "loading the token-skim kernels");
  WF_HIP(load_scan_kernels(), "loading the scan kernels");
  WF_HIP(load_attn_kernels(), "loading the attention kernels");
  WF_HIP(load_skim_kernels(), "loading the DWT and skim kernels");
  void* scratch_ptr = nullptr;  // this file's code object and its scratch array
  WF_TRY(scratch_of_current_device(&scratch_ptr));
  return ok();
}

const char* wf_status_str(wf_status s) {
  switch (s) {
    case WF_OK: return "WF_OK";
    case WF_ERR_INVALID_ARG: return "WF_ERR_INVALID_ARG";
    case WF_ERR_UNSUPPORTED: return "WF_ERR_UNSUPPORTED";
    case WF_ERR_WORKSPACE: return "WF_ERR_WORKSPACE";
    case WF_ERR_HIP: return "WF_ERR_HIP";
  }
  return "WF_ERR_UNKNOWN";
}

const char* wf_last_error(void) { return g_last_error; }

}  // extern "C"
