// C-ABI entry points of libdsattn.so: argument validation, threshold mapping and launch.
// Declared and documented in include/dsattn.h.

#include "dsattn.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>

#include "fa_fwd_launch.h"
#include "quant_launch.h"
#include "reorder_launch.h"

namespace {

thread_local std::string g_last_error;

constexpr int kHeadDim = 128;
constexpr int kTileQ = 128;
constexpr int kTileK = 64;
constexpr int kTileKPair = 128;  // one decision per two 64-key tiles
constexpr int kTileKHalf = 32;   // two decisions per 64-key tile
constexpr int kUnitWave = 32;  // tile_q = 32: each wave's 32 rows decide on their own
constexpr int kMaxMaskTiles = 4096;  // key tiles per head the mask-reuse kernel can list
constexpr double kLog2e = 1.4426950408889634074;

__attribute__((format(printf, 2, 3))) int fail(int code, const char* fmt, ...) {
  char buf[256];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

// True when `p` is memory the GPU can dereference (device or managed allocation).
bool is_device_pointer(const void* p) {
  hipPointerAttribute_t attr;
  const hipError_t e = hipPointerGetAttributes(&attr, p);
  if (e != hipSuccess) {
    (void)hipGetLastError();  // clear the sticky-free error state left by the query
    return false;
  }
  return attr.type == hipMemoryTypeDevice || attr.type == hipMemoryTypeManaged ||
         attr.type == hipMemoryTypeUnified;
}

struct Request {
  int rule;        // dsattn::kRule*
  float thr_log2;  // threshold in log2 units
};

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Size, scale and shape checks shared by every attention entry point.
int check_problem(const dsattn_args& a) {
  if (a.B < 0 || a.H < 0 || a.N < 0)
    return fail(DSATTN_EINVAL, "B, H and N must be >= 0");
  if (!(a.scale > 0.f) || !std::isfinite(a.scale))
    return fail(DSATTN_EINVAL, "scale must be finite and > 0 (got %g)", (double)a.scale);
  if (a.d != kHeadDim)
    return fail(DSATTN_EUNSUPPORTED, "head dimension %d is not supported (only 128)", a.d);
  if ((a.tile_q != kTileQ && a.tile_q != kUnitWave) ||
      (a.tile_k != kTileK && a.tile_k != kTileKPair && a.tile_k != kTileKHalf))
    return fail(DSATTN_EUNSUPPORTED,
                "tile shape %d x %d is not supported (tile_q 128 or 32, tile_k 32, 64 or 128)",
                a.tile_q, a.tile_k);
  const long long bh = (long long)a.B * (long long)a.H;
  if (bh > 65535) return fail(DSATTN_EINVAL, "B*H must be <= 65535 (got %lld)", bh);
  if ((long long)a.N * kHeadDim * bh > (1LL << 40))
    return fail(DSATTN_EINVAL, "problem too large");
  // The kernels address one head's keys and values (N rows of 256 bytes) through a
  // 32-bit buffer range.
  if ((long long)a.N * kHeadDim * 2 > INT32_MAX)
    return fail(DSATTN_EINVAL, "N must be <= %d (got %d)", (int)(INT32_MAX / (kHeadDim * 2)),
                a.N);
  if (a.key_order != DSATTN_ORDER_ASCENDING && a.key_order != DSATTN_ORDER_DIAGONAL)
    return fail(DSATTN_EINVAL, "unknown key order %d", a.key_order);
  if (a.qk_format != DSATTN_QK_BF16 && a.qk_format != DSATTN_QK_MXFP8)
    return fail(DSATTN_EINVAL, "unknown qk format %d", a.qk_format);
  if (a.qk_format == DSATTN_QK_MXFP8 && a.rule == DSATTN_RULE_MASK)
    return fail(DSATTN_EUNSUPPORTED, "mask reuse takes bf16 q and k");
  if (a.tile_k == kTileKHalf && a.key_order != DSATTN_ORDER_ASCENDING)
    return fail(DSATTN_EUNSUPPORTED, "tile_k = 32 visits key tiles in ascending order only");
  if (a.rule == DSATTN_RULE_MASK && a.tile_k == kTileKHalf)
    return fail(DSATTN_EUNSUPPORTED, "mask reuse takes tile_k = 64 or 128");
  if (a.rule == DSATTN_RULE_MASK) {
    if (a.key_order != DSATTN_ORDER_ASCENDING)
      return fail(DSATTN_EUNSUPPORTED, "mask reuse visits key tiles in ascending order only");
    if ((long long)a.N > (long long)kMaxMaskTiles * kTileK)
      return fail(DSATTN_EUNSUPPORTED, "mask reuse supports N <= %d (got %d)",
                  kMaxMaskTiles * kTileK, a.N);
  }
  return DSATTN_OK;
}

bool empty_problem(const dsattn_args& a) { return a.B == 0 || a.H == 0 || a.N == 0; }

// Byte ranges of the buffers one call reads and writes.
struct Span {
  const char* name;
  uintptr_t lo, hi;   // [lo, hi); empty when the buffer is absent
};

Span span(const char* name, const void* p, size_t bytes) {
  const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
  return Span{name, lo, p == nullptr ? lo : lo + bytes};
}

bool overlap(const Span& x, const Span& y) {
  return x.lo < x.hi && y.lo < y.hi && x.lo < y.hi && y.lo < x.hi;
}

// Byte ranges of the buffers one attention call reads (inputs) and writes (outputs).
struct CallSpans {
  Span in[6];
  Span out[4];
};

CallSpans call_spans(const dsattn_args& a) {
  const size_t rows = (size_t)a.B * (size_t)a.H * (size_t)a.N;
  const bool q8 = a.qk_format == DSATTN_QK_MXFP8;
  const size_t qk_bytes = rows * (size_t)kHeadDim * (q8 ? 1 : 2);
  const size_t units = (size_t)a.B * (size_t)a.H * (size_t)((a.N + a.tile_q - 1) / a.tile_q);
  const size_t mask_bytes = units * (size_t)((a.N + a.tile_k - 1) / a.tile_k);
  return CallSpans{
      {span("q", a.q, qk_bytes), span("k", a.k, qk_bytes), span("v", a.v, rows * kHeadDim * 2),
       span("q_scales", q8 ? a.q_scales : nullptr, rows * 4),
       span("k_scales", q8 ? a.k_scales : nullptr, rows * 4),
       span("mask_in", a.rule == DSATTN_RULE_MASK ? a.mask_in : nullptr, mask_bytes)},
      {span("o", a.o, rows * kHeadDim * 2), span("lse_out", a.lse_out, rows * 4),
       span("mask_out", a.mask_out, mask_bytes),
       span("stats_out", a.stats_out, (size_t)a.B * (size_t)a.H * 4 * sizeof(uint64_t))}};
}

// Every output must be disjoint from every input and from the other outputs (the kernels
// read inputs while writing outputs, from many workgroups at once).
int check_overlaps(const dsattn_args& a) {
  const CallSpans c = call_spans(a);
  for (const Span& w : c.out) {
    for (const Span& r : c.in)
      if (overlap(w, r)) return fail(DSATTN_EINVAL, "%s must not overlap %s", w.name, r.name);
    for (const Span& w2 : c.out)
      if (&w2 < &w && overlap(w, w2))
        return fail(DSATTN_EINVAL, "%s must not overlap %s", w.name, w2.name);
  }
  return DSATTN_OK;
}

// Pointer checks of a non-empty problem.
int check_pointers(const dsattn_args& a) {
  if (a.q == nullptr || a.k == nullptr || a.v == nullptr || a.o == nullptr)
    return fail(DSATTN_EINVAL, "q, k, v and o must be non-null");
  const void* ptrs[] = {a.q, a.k, a.v, a.o};
  const char* names[] = {"q", "k", "v", "o"};
  for (int i = 0; i < 4; ++i) {
    if (!is_device_pointer(ptrs[i]))
      return fail(DSATTN_EINVAL, "%s is not a device pointer", names[i]);
    if (!aligned(ptrs[i], 16))
      return fail(DSATTN_EINVAL, "%s must be 16-byte aligned", names[i]);
  }
  if (a.stats_out != nullptr && !is_device_pointer(a.stats_out))
    return fail(DSATTN_EINVAL, "stats_out is not a device pointer");
  if (a.mask_out != nullptr && !is_device_pointer(a.mask_out))
    return fail(DSATTN_EINVAL, "mask_out is not a device pointer");
  if (a.lse_out != nullptr && !is_device_pointer(a.lse_out))
    return fail(DSATTN_EINVAL, "lse_out is not a device pointer");
  if (a.lse_out != nullptr && !aligned(a.lse_out, 4))
    return fail(DSATTN_EINVAL, "lse_out must be 4-byte aligned");
  if (a.qk_format == DSATTN_QK_MXFP8) {
    if (a.q_scales == nullptr || a.k_scales == nullptr)
      return fail(DSATTN_EINVAL, "MX-FP8 q and k need q_scales and k_scales");
    if (!is_device_pointer(a.q_scales) || !is_device_pointer(a.k_scales))
      return fail(DSATTN_EINVAL, "q_scales and k_scales must be device pointers");
    if (!aligned(a.q_scales, 4) || !aligned(a.k_scales, 4))
      return fail(DSATTN_EINVAL, "q_scales and k_scales must be 4-byte aligned");
  }
  if (a.rule == DSATTN_RULE_MASK) {
    if (a.mask_in == nullptr) return fail(DSATTN_EINVAL, "mask reuse needs mask_in");
    if (!is_device_pointer(a.mask_in)) return fail(DSATTN_EINVAL, "mask_in is not a device pointer");
  }
  return check_overlaps(a);
}

// Zero stats_out of an empty problem (the only output it has).
int finish_empty(const dsattn_args& a) {
  const long long bh = (long long)a.B * (long long)a.H;
  if (a.stats_out != nullptr && bh > 0) {
    if (!is_device_pointer(a.stats_out))
      return fail(DSATTN_EINVAL, "stats_out is not a device pointer");
    if (dsattn::launch_zero_u64(a.stats_out, (int)(bh * 4), a.stream) != hipSuccess)
      return fail(DSATTN_ELAUNCH, "zero-fill launch failed");
  }
  g_last_error.clear();
  return DSATTN_OK;
}

// Enqueue the attention kernels of a checked, non-empty problem.
int launch_attention(const dsattn_args& a, const Request& rq) {
  const long long bh = (long long)a.B * (long long)a.H;
  dsattn::FwdParams p;
  p.q = static_cast<const uint16_t*>(a.q);
  p.k = static_cast<const uint16_t*>(a.k);
  p.v = static_cast<const uint16_t*>(a.v);
  p.o = static_cast<uint16_t*>(a.o);
  p.N = a.N;
  p.n_qt = (a.N + kTileQ - 1) / kTileQ;
  p.n_qu = (a.N + a.tile_q - 1) / a.tile_q;
  p.n_kt = (a.N + kTileK - 1) / kTileK;
  p.c = (float)((double)a.scale * kLog2e);
  p.thr = rq.thr_log2;
  p.stats = a.stats_out;
  p.mask = a.mask_out;
  p.lse = a.lse_out;
  p.key_order = a.key_order == DSATTN_ORDER_DIAGONAL ? dsattn::kOrderDiagonal
                                                     : dsattn::kOrderAscending;
  p.mask_in = a.rule == DSATTN_RULE_MASK ? a.mask_in : nullptr;
  p.key_tile = a.tile_k;
  p.n_kd = (a.N + a.tile_k - 1) / a.tile_k;
  const bool q8 = a.qk_format == DSATTN_QK_MXFP8;
  p.qk_format = q8 ? dsattn::kQkMxfp8 : dsattn::kQkBf16;
  p.q8 = q8 ? static_cast<const uint8_t*>(a.q) : nullptr;
  p.k8 = q8 ? static_cast<const uint8_t*>(a.k) : nullptr;
  p.q_scales = q8 ? a.q_scales : nullptr;
  p.k_scales = q8 ? a.k_scales : nullptr;
  if (q8) p.q = p.k = nullptr;

  if (p.stats != nullptr &&
      dsattn::launch_zero_u64(p.stats, (int)(bh * 4), a.stream) != hipSuccess)
    return fail(DSATTN_ELAUNCH, "zero-fill launch failed");
  const hipError_t e = dsattn::launch_fa_fwd(rq.rule, a.tile_q, p, (int)bh, a.stream);
  if (e != hipSuccess) return fail(DSATTN_ELAUNCH, "kernel launch failed: %s", hipGetErrorString(e));
  return DSATTN_OK;
}

int run(const dsattn_args& a, const Request& rq) {
  int rc = check_problem(a);
  if (rc != DSATTN_OK) return rc;
  if (empty_problem(a)) return finish_empty(a);
  if ((rc = check_pointers(a)) != DSATTN_OK) return rc;
  if ((rc = launch_attention(a, rq)) != DSATTN_OK) return rc;
  g_last_error.clear();
  return DSATTN_OK;
}

// ---- token reordering -----------------------------------------------------------------

// True unless `p` is device-only memory (the host writes the block order directly).
bool host_writable(const void* p) {
  hipPointerAttribute_t attr;
  if (hipPointerGetAttributes(&attr, p) != hipSuccess) {
    (void)hipGetLastError();
    return true;  // ordinary pageable host memory is unknown to the runtime
  }
  return attr.type != hipMemoryTypeDevice;
}

// Checks of a row move over [bh][N][row_bytes]; sets *wide when 16-byte chunks can be used.
int check_rows(const void* src, const void* dst, const int32_t* index, int bh, int N,
               int row_bytes, bool* wide) {
  if (bh < 0 || N < 0) return fail(DSATTN_EINVAL, "BH and N must be >= 0");
  if (bh > 65535) return fail(DSATTN_EINVAL, "BH must be <= 65535 (got %d)", bh);
  if (row_bytes <= 0 || row_bytes % 4 != 0)
    return fail(DSATTN_EINVAL, "row_bytes must be a positive multiple of 4 (got %d)", row_bytes);
  if ((long long)N * (row_bytes / 4) > (1LL << 31))
    return fail(DSATTN_EINVAL, "N * row_bytes is too large for one head");
  if (bh == 0 || N == 0) return DSATTN_OK;
  if (src == nullptr || dst == nullptr || index == nullptr)
    return fail(DSATTN_EINVAL, "src, dst and index must be non-null");
  const void* ptrs[] = {src, dst, index};
  const char* names[] = {"src", "dst", "index"};
  for (int i = 0; i < 3; ++i) {
    if (!is_device_pointer(ptrs[i]))
      return fail(DSATTN_EINVAL, "%s is not a device pointer", names[i]);
    if (!aligned(ptrs[i], 4)) return fail(DSATTN_EINVAL, "%s must be 4-byte aligned", names[i]);
  }
  const uintptr_t bytes = (uintptr_t)bh * (uintptr_t)N * (uintptr_t)row_bytes;
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
  if (s0 < d0 + bytes && d0 < s0 + bytes)
    return fail(DSATTN_EINVAL, "src and dst must not overlap");
  *wide = row_bytes % 16 == 0 && aligned(src, 16) && aligned(dst, 16);
  return DSATTN_OK;
}

constexpr size_t kSliceAlign = 256;

size_t round_up(size_t x) { return (x + kSliceAlign - 1) / kSliceAlign * kSliceAlign; }

size_t workspace_bytes(int B, int H, int N, int d, bool with_lse) {
  if (B <= 0 || H <= 0 || N <= 0 || d <= 0) return 0;
  const size_t bhn = (size_t)B * (size_t)H * (size_t)N;
  const size_t slice = round_up(bhn * (size_t)d * 2);
  return 4 * slice + (with_lse ? round_up(bhn * 4) : 0);
}

double lambda_from_recall(double r, int n) {
  if (!(r > 0.0 && r <= 1.0) || n <= 0) return std::nan("");
  if (r == 1.0) return -INFINITY;
  return std::log((1.0 - r) / (double)n);
}

int resolve_request(const dsattn_args& a, Request* rq) {
  switch (a.rule) {
    case DSATTN_RULE_DENSE:
      rq->rule = dsattn::kRuleDense;
      rq->thr_log2 = -INFINITY;
      return DSATTN_OK;
    case DSATTN_RULE_BLASST: {
      const float tau = a.param;
      if (!(tau >= 0.f && tau <= 1.f))
        return fail(DSATTN_EINVAL, "BLASST threshold tau must lie in [0, 1] (got %g)", (double)tau);
      rq->rule = dsattn::kRuleBlasst;
      rq->thr_log2 = tau == 0.f ? -INFINITY : (float)std::log2((double)tau);
      return DSATTN_OK;
    }
    case DSATTN_RULE_DYNSPARSE_RECALL: {
      const float r = a.param;
      if (!(r > 0.f && r <= 1.f))
        return fail(DSATTN_EINVAL, "recall target must lie in (0, 1] (got %g)", (double)r);
      rq->rule = dsattn::kRuleDynSparse;
      const double lam = a.N > 0 ? lambda_from_recall(r, a.N) : -INFINITY;
      rq->thr_log2 = (float)(lam * kLog2e);
      return DSATTN_OK;
    }
    case DSATTN_RULE_MASK:
      rq->rule = dsattn::kRuleMask;
      rq->thr_log2 = 0.f;
      return DSATTN_OK;
    case DSATTN_RULE_DYNSPARSE_LAMBDA: {
      const float lam = a.param;
      if (std::isnan(lam) || lam == INFINITY)
        return fail(DSATTN_EINVAL, "lambda must be finite or -inf (got %g)", (double)lam);
      rq->rule = dsattn::kRuleDynSparse;
      rq->thr_log2 = (float)((double)lam * kLog2e);
      return DSATTN_OK;
    }
    default:
      return fail(DSATTN_EINVAL, "unknown rule %d", a.rule);
  }
}

dsattn_args make_args(int rule, float param, const void* q, const void* k, const void* v,
                      void* o, int B, int H, int N, int d, float scale, int tile_q,
                      int tile_k, hipStream_t stream, uint64_t* stats_out) {
  dsattn_args a;
  a.rule = rule;
  a.param = param;
  a.q = q;
  a.k = k;
  a.v = v;
  a.o = o;
  a.B = B;
  a.H = H;
  a.N = N;
  a.d = d;
  a.scale = scale;
  a.tile_q = tile_q;
  a.tile_k = tile_k;
  a.stream = stream;
  a.stats_out = stats_out;
  a.mask_out = nullptr;
  a.lse_out = nullptr;
  a.key_order = DSATTN_ORDER_ASCENDING;
  a.mask_in = nullptr;
  a.qk_format = DSATTN_QK_BF16;
  a.q_scales = nullptr;
  a.k_scales = nullptr;
  return a;
}

}  // namespace

extern "C" {

float dsattn_lambda_from_recall(float recall_target, int N) {
  return (float)lambda_from_recall(recall_target, N);
}

int dsattn_attn_fwd_ex(const dsattn_args* args) {
  if (args == nullptr) return fail(DSATTN_EINVAL, "args must be non-null");
  Request rq;
  const int rc = resolve_request(*args, &rq);
  if (rc != DSATTN_OK) return rc;
  return run(*args, rq);
}

int dynsparse_attn_fwd(const void* q, const void* k, const void* v, void* o, int B, int H,
                       int N, int d, float scale, float recall_target, int tile_q, int tile_k,
                       hipStream_t stream, uint64_t* stats_out) {
  const dsattn_args a = make_args(DSATTN_RULE_DYNSPARSE_RECALL, recall_target, q, k, v, o, B,
                                  H, N, d, scale, tile_q, tile_k, stream, stats_out);
  return dsattn_attn_fwd_ex(&a);
}

int dynsparse_attn_fwd_lambda(const void* q, const void* k, const void* v, void* o, int B,
                              int H, int N, int d, float scale, float lambda, int tile_q,
                              int tile_k, hipStream_t stream, uint64_t* stats_out) {
  const dsattn_args a = make_args(DSATTN_RULE_DYNSPARSE_LAMBDA, lambda, q, k, v, o, B, H, N,
                                  d, scale, tile_q, tile_k, stream, stats_out);
  return dsattn_attn_fwd_ex(&a);
}

int blasst_attn_fwd(const void* q, const void* k, const void* v, void* o, int B, int H, int N,
                    int d, float scale, float threshold, int tile_q, int tile_k,
                    hipStream_t stream, uint64_t* stats_out) {
  const dsattn_args a = make_args(DSATTN_RULE_BLASST, threshold, q, k, v, o, B, H, N, d, scale,
                                  tile_q, tile_k, stream, stats_out);
  return dsattn_attn_fwd_ex(&a);
}

int dense_attn_fwd(const void* q, const void* k, const void* v, void* o, int B, int H, int N,
                   int d, float scale, int tile_q, int tile_k, hipStream_t stream,
                   uint64_t* stats_out) {
  const dsattn_args a = make_args(DSATTN_RULE_DENSE, 0.f, q, k, v, o, B, H, N, d, scale,
                                  tile_q, tile_k, stream, stats_out);
  return dsattn_attn_fwd_ex(&a);
}

int dsattn_block_order(int T, int Y, int X, int bt, int by, int bx, int32_t* perm_out) {
  if (T <= 0 || Y <= 0 || X <= 0 || bt <= 0 || by <= 0 || bx <= 0)
    return fail(DSATTN_EINVAL, "grid and block extents must be positive");
  const long long n = (long long)T * Y * X;
  if (n > 0x7fffffffLL) return fail(DSATTN_EINVAL, "grid has more than 2^31 - 1 tokens");
  if (perm_out == nullptr) return fail(DSATTN_EINVAL, "perm_out must be non-null");
  if (!host_writable(perm_out)) return fail(DSATTN_EINVAL, "perm_out must be host memory");
  // The reordered position of token (t, y, x) in closed form: the tokens of all earlier
  // block slabs along t, then of the earlier block rows of its slab, then of the earlier
  // blocks of its block row, then its row-major rank inside its own (possibly clipped)
  // block.
  const long long YX = (long long)Y * X;
  for (int t = 0; t < T; ++t) {
    const int t0 = t / bt * bt, et = std::min(bt, T - t0);
    for (int y = 0; y < Y; ++y) {
      const int y0 = y / by * by, ey = std::min(by, Y - y0);
      for (int x = 0; x < X; ++x) {
        const int x0 = x / bx * bx, ex = std::min(bx, X - x0);
        const long long pos = (long long)t0 * YX + (long long)et * y0 * X +
                              (long long)et * ey * x0 +
                              ((long long)(t - t0) * ey + (y - y0)) * ex + (x - x0);
        perm_out[pos] = (int32_t)((long long)t * YX + (long long)y * X + x);
      }
    }
  }
  g_last_error.clear();
  return DSATTN_OK;
}

int dsattn_gather_rows(const void* src, void* dst, const int32_t* index, int BH, int N,
                       int row_bytes, hipStream_t stream) {
  bool wide = false;
  const int rc = check_rows(src, dst, index, BH, N, row_bytes, &wide);
  if (rc != DSATTN_OK) return rc;
  if (BH > 0 && N > 0) {
    const hipError_t e = dsattn::launch_gather_rows(src, dst, index, BH, N, row_bytes, wide, stream);
    if (e != hipSuccess) return fail(DSATTN_ELAUNCH, "gather launch failed: %s", hipGetErrorString(e));
  }
  g_last_error.clear();
  return DSATTN_OK;
}

int dsattn_scatter_rows(const void* src, void* dst, const int32_t* index, int BH, int N,
                        int row_bytes, hipStream_t stream) {
  bool wide = false;
  const int rc = check_rows(src, dst, index, BH, N, row_bytes, &wide);
  if (rc != DSATTN_OK) return rc;
  if (BH > 0 && N > 0) {
    const hipError_t e = dsattn::launch_scatter_rows(src, dst, index, BH, N, row_bytes, wide, stream);
    if (e != hipSuccess) return fail(DSATTN_ELAUNCH, "scatter launch failed: %s", hipGetErrorString(e));
  }
  g_last_error.clear();
  return DSATTN_OK;
}

size_t dsattn_reordered_workspace_bytes(int B, int H, int N, int d, int with_lse) {
  return workspace_bytes(B, H, N, d, with_lse != 0);
}

}  // extern "C"

namespace {

// Reordered attention over a workspace of workspace_size bytes.  static_ws: the workspace
// is the library's own static scratch (device memory by construction; its size is the
// fixed maximum).
int reordered(const dsattn_args* args, const int32_t* q_index, const int32_t* kv_index,
              void* workspace, size_t workspace_size, bool static_ws) {
  if (args == nullptr) return fail(DSATTN_EINVAL, "args must be non-null");
  const dsattn_args& a = *args;
  Request rq;
  int rc = resolve_request(a, &rq);
  if (rc != DSATTN_OK) return rc;
  if ((rc = check_problem(a)) != DSATTN_OK) return rc;
  if (a.qk_format != DSATTN_QK_BF16)
    return fail(DSATTN_EUNSUPPORTED, "the reordered entry point takes bf16 q and k");
  if (empty_problem(a)) return finish_empty(a);
  if ((rc = check_pointers(a)) != DSATTN_OK) return rc;
  if (q_index == nullptr || kv_index == nullptr || workspace == nullptr)
    return fail(DSATTN_EINVAL, "q_index, kv_index and workspace must be non-null");
  if (!is_device_pointer(q_index) || !is_device_pointer(kv_index))
    return fail(DSATTN_EINVAL, "q_index and kv_index must be device pointers");
  if (!aligned(q_index, 4) || !aligned(kv_index, 4))
    return fail(DSATTN_EINVAL, "q_index and kv_index must be 4-byte aligned");
  if (!static_ws && !is_device_pointer(workspace))
    return fail(DSATTN_EINVAL, "workspace is not a device pointer");
  if (!aligned(workspace, kSliceAlign))
    return fail(DSATTN_EINVAL, "workspace must be %zu-byte aligned", kSliceAlign);
  const bool with_lse = a.lse_out != nullptr;
  const size_t need = workspace_bytes(a.B, a.H, a.N, a.d, with_lse);
  if (workspace_size < need) {
    if (static_ws)
      return fail(DSATTN_EINVAL,
                  "problem too large for the static scratch: %zu bytes needed, %zu available "
                  "(use dsattn_attn_fwd_reordered with a caller workspace)",
                  need, workspace_size);
    return fail(DSATTN_EINVAL, "workspace too small: %zu bytes given, %zu needed", workspace_size, need);
  }

  // The gathers read q, k, v and the index arrays into the workspace, the kernel reads
  // and writes the workspace while writing mask_out and stats_out, and the scatters read
  // the workspace and q_index into o and lse_out: the workspace must be disjoint from
  // every argument buffer, and the index arrays from everything written.
  const CallSpans c = call_spans(a);
  const Span ws_span = span("workspace", workspace, need);
  const Span idx[] = {span("q_index", q_index, (size_t)a.N * 4),
                      span("kv_index", kv_index, (size_t)a.N * 4)};
  for (const Span& r : c.in)
    if (overlap(ws_span, r)) return fail(DSATTN_EINVAL, "workspace must not overlap %s", r.name);
  for (const Span& w : c.out)
    if (overlap(ws_span, w)) return fail(DSATTN_EINVAL, "workspace must not overlap %s", w.name);
  for (const Span& i : idx) {
    if (overlap(ws_span, i)) return fail(DSATTN_EINVAL, "workspace must not overlap %s", i.name);
    for (const Span& w : c.out)
      if (overlap(w, i)) return fail(DSATTN_EINVAL, "%s must not overlap %s", w.name, i.name);
  }
  const int bh = a.B * a.H;
  const size_t slice = round_up((size_t)bh * (size_t)a.N * (size_t)a.d * 2);
  char* ws = static_cast<char*>(workspace);
  dsattn_args r = a;  // the same problem over the reordered sequence
  r.q = ws;
  r.k = ws + slice;
  r.v = ws + 2 * slice;
  r.o = ws + 3 * slice;
  r.lse_out = with_lse ? reinterpret_cast<float*>(ws + 4 * slice) : nullptr;
  const int row = a.d * 2;
  const struct {
    const void* src;
    const void* dst;
    const int32_t* index;
  } gathers[] = {{a.q, r.q, q_index}, {a.k, r.k, kv_index}, {a.v, r.v, kv_index}};
  for (const auto& g : gathers) {
    const hipError_t e = dsattn::launch_gather_rows(g.src, const_cast<void*>(g.dst), g.index, bh,
                                                    a.N, row, true, a.stream);
    if (e != hipSuccess) return fail(DSATTN_ELAUNCH, "gather launch failed: %s", hipGetErrorString(e));
  }
  if ((rc = launch_attention(r, rq)) != DSATTN_OK) return rc;
  hipError_t e = dsattn::launch_scatter_rows(r.o, a.o, q_index, bh, a.N, row, true, a.stream);
  if (e == hipSuccess && with_lse)
    e = dsattn::launch_scatter_rows(r.lse_out, a.lse_out, q_index, bh, a.N, 4, false, a.stream);
  if (e != hipSuccess) return fail(DSATTN_ELAUNCH, "scatter launch failed: %s", hipGetErrorString(e));
  g_last_error.clear();
  return DSATTN_OK;
}

// Scratch of the allocation-free reordered entry point: one copy per GPU, held until the
// process ends.  Host code never names the array itself (on the host its name is only a
// stand-in); it uses the device address hipGetSymbolAddress returns for the current
// device, looked up once per device on the first call there.
constexpr size_t kStaticScratchBytes = DSATTN_STATIC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
static __device__ __attribute__((aligned(256))) unsigned char scratch[kStaticScratchBytes];

std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

int static_scratch(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return fail(DSATTN_EINVAL, "no usable current HIP device");
  }
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return fail(DSATTN_ELAUNCH, "static scratch lookup failed on device %d: %s", dev,
                  hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return DSATTN_OK;
}

}  // namespace

extern "C" {

int dsattn_attn_fwd_reordered(const dsattn_args* args, const int32_t* q_index,
                              const int32_t* kv_index, void* workspace,
                              size_t workspace_size) {
  return reordered(args, q_index, kv_index, workspace, workspace_size, false);
}

int dsattn_attn_fwd_reordered_noalloc(const dsattn_args* args, const int32_t* q_index,
                                      const int32_t* kv_index) {
  if (args == nullptr) return fail(DSATTN_EINVAL, "args must be non-null");
  void* ws = nullptr;
  // an empty problem touches no scratch
  if (args->B != 0 && args->H != 0 && args->N != 0) {
    const int rc = static_scratch(&ws);
    if (rc != DSATTN_OK) return rc;
  }
  return reordered(args, q_index, kv_index, ws, kStaticScratchBytes, true);
}

namespace {

int quantize(const void* src, const float* shift, void* codes, void* scales, long long rows,
             int row_len, long long group_rows, hipStream_t stream) {
  if (rows < 0) return fail(DSATTN_EINVAL, "rows must be >= 0");
  if (row_len <= 0 || row_len % 32 != 0)
    return fail(DSATTN_EINVAL, "row_len must be a positive multiple of 32 (got %d)", row_len);
  if (shift != nullptr && group_rows <= 0)
    return fail(DSATTN_EINVAL, "group_rows must be > 0 (got %lld)", group_rows);
  const long long n_blocks = rows * (row_len / 32);
  if (rows > 0 && n_blocks / rows != row_len / 32) return fail(DSATTN_EINVAL, "problem too large");
  // one thread per block, 256 per workgroup: keep the grid far inside its 2^31 limit
  if (n_blocks > (1LL << 36)) return fail(DSATTN_EINVAL, "problem too large");
  if (n_blocks == 0) {
    g_last_error.clear();
    return DSATTN_OK;
  }
  const void* ptrs[] = {src, codes, scales};
  const char* names[] = {"src", "codes", "scales"};
  for (int i = 0; i < 3; ++i) {
    if (ptrs[i] == nullptr) return fail(DSATTN_EINVAL, "%s must be non-null", names[i]);
    if (!is_device_pointer(ptrs[i]))
      return fail(DSATTN_EINVAL, "%s is not a device pointer", names[i]);
  }
  if (!aligned(src, 16) || !aligned(codes, 16))
    return fail(DSATTN_EINVAL, "src and codes must be 16-byte aligned");
  if (shift != nullptr && (!is_device_pointer(shift) || !aligned(shift, 16)))
    return fail(DSATTN_EINVAL, "shift must be a 16-byte aligned device pointer");
  const hipError_t e = dsattn::launch_quantize_mxfp8(src, codes, scales, n_blocks, shift,
                                                     row_len / 32, group_rows, stream);
  if (e != hipSuccess) return fail(DSATTN_ELAUNCH, "quantize launch failed: %s", hipGetErrorString(e));
  g_last_error.clear();
  return DSATTN_OK;
}

}  // namespace

int dsattn_quantize_mxfp8(const void* src, void* codes, void* scales, long long rows,
                          int row_len, hipStream_t stream) {
  return quantize(src, nullptr, codes, scales, rows, row_len, 1, stream);
}

int dsattn_quantize_mxfp8_shift(const void* src, const float* shift, void* codes, void* scales,
                                long long rows, int row_len, long long group_rows,
                                hipStream_t stream) {
  if (shift == nullptr) return fail(DSATTN_EINVAL, "shift must be non-null");
  return quantize(src, shift, codes, scales, rows, row_len, group_rows, stream);
}

int dsattn_key_mean(const void* k, float* mean_out, int BH, int N, int d, hipStream_t stream) {
  if (BH < 0 || N < 0) return fail(DSATTN_EINVAL, "BH and N must be >= 0");
  if (BH > 65535) return fail(DSATTN_EINVAL, "BH must be <= 65535 (got %d)", BH);
  if (d < 8 || d > 1024 || (d & (d - 1)) != 0)
    return fail(DSATTN_EINVAL, "d must be a power of two in [8, 1024] (got %d)", d);
  if (N == 0 || BH == 0) {
    if (N == 0 && BH > 0) return fail(DSATTN_EINVAL, "the mean of zero keys is undefined");
    g_last_error.clear();
    return DSATTN_OK;
  }
  if ((long long)N * d > (1LL << 31)) return fail(DSATTN_EINVAL, "N * d is too large for one head");
  if (k == nullptr || mean_out == nullptr) return fail(DSATTN_EINVAL, "k and mean_out must be non-null");
  if (!is_device_pointer(k) || !is_device_pointer(mean_out))
    return fail(DSATTN_EINVAL, "k and mean_out must be device pointers");
  if (!aligned(k, 16) || !aligned(mean_out, 4))
    return fail(DSATTN_EINVAL, "k must be 16-byte and mean_out 4-byte aligned");
  const hipError_t e = dsattn::launch_key_mean(k, mean_out, BH, N, d, stream);
  if (e != hipSuccess) return fail(DSATTN_ELAUNCH, "key mean launch failed: %s", hipGetErrorString(e));
  g_last_error.clear();
  return DSATTN_OK;
}

const char* dsattn_last_error(void) { return g_last_error.c_str(); }

const char* dsattn_version(void) { return "dsattn 0.1 (gfx950)"; }

}  // extern "C"
