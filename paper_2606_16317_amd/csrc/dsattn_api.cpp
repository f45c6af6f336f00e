// C-ABI entry points of libdsattn.so: argument validation, threshold mapping and launch.
// Declared and documented in include/dsattn.h.

#include "dsattn.h"

#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>

#include "fa_fwd_launch.h"

namespace {

thread_local std::string g_last_error;

constexpr int kHeadDim = 128;
constexpr int kTileQ = 128;
constexpr int kTileK = 64;
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

int run(const dsattn_args& a, const Request& rq) {
  if (a.B < 0 || a.H < 0 || a.N < 0)
    return fail(DSATTN_EINVAL, "B, H and N must be >= 0");
  if (!(a.scale > 0.f) || !std::isfinite(a.scale))
    return fail(DSATTN_EINVAL, "scale must be finite and > 0 (got %g)", (double)a.scale);
  if (a.d != kHeadDim)
    return fail(DSATTN_EUNSUPPORTED, "head dimension %d is not supported (only 128)", a.d);
  if (a.tile_q != kTileQ || a.tile_k != kTileK)
    return fail(DSATTN_EUNSUPPORTED, "tile shape %d x %d is not supported (only 128 x 64)", a.tile_q, a.tile_k);
  const long long bh = (long long)a.B * (long long)a.H;
  if (bh > 65535) return fail(DSATTN_EINVAL, "B*H must be <= 65535 (got %lld)", bh);
  if ((long long)a.N * kHeadDim * bh > (1LL << 40))
    return fail(DSATTN_EINVAL, "problem too large");

  if (bh == 0 || a.N == 0) {
    if (a.stats_out != nullptr && bh > 0) {
      if (!is_device_pointer(a.stats_out))
        return fail(DSATTN_EINVAL, "stats_out is not a device pointer");
      if (dsattn::launch_zero_u64(a.stats_out, (int)(bh * 4), a.stream) != hipSuccess)
        return fail(DSATTN_ELAUNCH, "zero-fill launch failed");
    }
    g_last_error.clear();
    return DSATTN_OK;
  }
  if (a.q == nullptr || a.k == nullptr || a.v == nullptr || a.o == nullptr)
    return fail(DSATTN_EINVAL, "q, k, v and o must be non-null");
  const void* ptrs[] = {a.q, a.k, a.v, a.o};
  const char* names[] = {"q", "k", "v", "o"};
  for (int i = 0; i < 4; ++i)
    if (!is_device_pointer(ptrs[i]))
      return fail(DSATTN_EINVAL, "%s is not a device pointer", names[i]);
  if (a.o == a.q || a.o == a.k || a.o == a.v)
    return fail(DSATTN_EINVAL, "o must not alias q, k or v");
  if (a.stats_out != nullptr && !is_device_pointer(a.stats_out))
    return fail(DSATTN_EINVAL, "stats_out is not a device pointer");
  if (a.mask_out != nullptr && !is_device_pointer(a.mask_out))
    return fail(DSATTN_EINVAL, "mask_out is not a device pointer");
  if (a.lse_out != nullptr && !is_device_pointer(a.lse_out))
    return fail(DSATTN_EINVAL, "lse_out is not a device pointer");

  dsattn::FwdParams p;
  p.q = static_cast<const uint16_t*>(a.q);
  p.k = static_cast<const uint16_t*>(a.k);
  p.v = static_cast<const uint16_t*>(a.v);
  p.o = static_cast<uint16_t*>(a.o);
  p.N = a.N;
  p.n_qt = (a.N + kTileQ - 1) / kTileQ;
  p.n_kt = (a.N + kTileK - 1) / kTileK;
  p.c = (float)((double)a.scale * kLog2e);
  p.thr = rq.thr_log2;
  p.stats = a.stats_out;
  p.mask = a.mask_out;
  p.lse = a.lse_out;

  if (p.stats != nullptr &&
      dsattn::launch_zero_u64(p.stats, (int)(bh * 4), a.stream) != hipSuccess)
    return fail(DSATTN_ELAUNCH, "zero-fill launch failed");
  const hipError_t e = dsattn::launch_fa_fwd(rq.rule, p, (int)bh, a.stream);
  if (e != hipSuccess) return fail(DSATTN_ELAUNCH, "kernel launch failed: %s", hipGetErrorString(e));
  g_last_error.clear();
  return DSATTN_OK;
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

const char* dsattn_last_error(void) { return g_last_error.c_str(); }

const char* dsattn_version(void) { return "dsattn 0.1 (gfx950)"; }

}  // extern "C"
