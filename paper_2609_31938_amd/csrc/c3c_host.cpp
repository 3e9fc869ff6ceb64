// C-ABI host layer of libc3c: validation, the temporal-interval algebra of
// Eq. 3 / Eq. 4, the route predicate (the guard of Alg. 1 plus the fast
// kernel's specialisation), route counters and the fallback-shape histogram,
// modes, and dispatch to the kernels on the caller's stream.
//
// Everything before a kernel launch is plain host code: route queries, output
// sizes, strict-mode rejections and argument errors never touch the device.
// The split-K plan (workspace size, plan query) reads the current device's
// compute-unit count, once per device.
#include <hip/hip_runtime.h>

#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "c3c.h"
#include "c3c_internal.h"

struct c3c_ctx {
  uint32_t mode = 0;
  c3c_counters ctr{};
  std::vector<c3c_sig_count> shapes;
  std::string last_error;
  void* ws = nullptr;      // caller's split-K workspace (device memory)
  size_t ws_bytes = 0;
};

namespace c3c {
namespace {

constexpr uint32_t kModeMask =
    C3C_MODE_STRICT | C3C_MODE_FORCE_FALLBACK | C3C_MODE_INJECT_FAST_FAILURE |
    C3C_MODE_CHANNEL_TILES;
constexpr int64_t kMaxElems = int64_t(1) << 40;  // per tensor, far above any HBM size

int64_t floordiv(int64_t a, int64_t b) {
  int64_t q = a / b;
  if ((a % b != 0) && ((a < 0) != (b < 0))) --q;
  return q;
}

// Eq. 3 for time; the same closed form for a spatial axis with symmetric pad.
int64_t out_len(int64_t in, int64_t lo, int64_t hi, int64_t dil, int64_t k, int64_t stride) {
  return floordiv(in + lo + hi - dil * (k - 1) - 1, stride) + 1;
}

int elem_bytes(int32_t dtype) {
  switch (dtype) {
    case C3C_DTYPE_BF16: return 2;
    case C3C_DTYPE_F16: return 2;
    case C3C_DTYPE_F32: return 4;
    default: return 0;
  }
}

bool mul_ok(int64_t a, int64_t b, int64_t* out) {
  if (a < 0 || b < 0) return false;
  if (a != 0 && b > kMaxElems / a) return false;
  *out = a * b;
  return true;
}

// Validates the descriptor and fills the geometry.  Returns an empty string
// on success, else the reason it is invalid.
const char* make_geo(const c3c_conv_desc* d, Geo* g) {
  if (!d) return "descriptor is NULL";
  if (d->N < 1 || d->Ci < 1 || d->Co < 1 || d->H < 1 || d->W < 1)
    return "N, Ci, Co, H, W must be >= 1";
  if (d->Kt < 1 || d->Kh < 1 || d->Kw < 1) return "kernel sizes must be >= 1";
  if (d->T < 0 || d->Tc < 0) return "T and Tc must be >= 0";
  if (d->stride_t < 1 || d->stride_h < 1 || d->stride_w < 1) return "strides must be >= 1";
  if (d->dil_t < 1 || d->dil_h < 1 || d->dil_w < 1) return "dilations must be >= 1";
  if (d->pad_t_base < 0 || d->pad_h < 0 || d->pad_w < 0) return "pads must be >= 0";
  if (d->groups < 1 || d->Ci % d->groups || d->Co % d->groups)
    return "groups must divide Ci and Co";
  if (!elem_bytes(d->dtype)) return "unknown dtype";
  if (d->has_bias != 0 && d->has_bias != 1) return "has_bias must be 0 or 1";
  const int64_t big = int64_t(1) << 31;
  if (d->N >= big || d->Ci >= big || d->Co >= big || d->T >= big || d->Tc >= big ||
      d->H >= big || d->W >= big || d->Kt >= big || d->Kh >= big || d->Kw >= big ||
      d->pad_t_base >= big || d->pad_t_right >= big || -d->pad_t_right >= big ||
      d->pad_h >= big || d->pad_w >= big || d->stride_t >= big || d->stride_h >= big ||
      d->stride_w >= big || d->dil_t >= big || d->dil_h >= big || d->dil_w >= big)
    return "a size exceeds 2^31";
  g->d = *d;
  g->Z = d->Tc + d->T;
  g->p_l = d->pad_t_base - d->Tc;
  const int64_t to = out_len(g->Z, g->p_l, d->pad_t_right, d->dil_t, d->Kt, d->stride_t);
  g->To = to < 0 ? 0 : to;
  g->Ho = out_len(d->H, d->pad_h, d->pad_h, d->dil_h, d->Kh, d->stride_h);
  g->Wo = out_len(d->W, d->pad_w, d->pad_w, d->dil_w, d->Kw, d->stride_w);
  if (g->Ho < 1 || g->Wo < 1) return "spatial output would be empty";
  g->L = d->pad_t_base < g->Z ? d->pad_t_base : g->Z;
  g->elem = elem_bytes(d->dtype);
  if (d->H * d->W * g->elem >= big || g->Ho * g->Wo * g->elem >= big)
    return "a frame plane exceeds 2^31 bytes";
  int64_t t;
  if (!mul_ok(d->N * d->Ci, g->Z, &t) || !mul_ok(t, d->H * d->W, &t)) return "input too large";
  if (!mul_ok(d->N * d->Co, g->To, &t) || !mul_ok(t, g->Ho * g->Wo, &t)) return "output too large";
  if (!mul_ok(d->Co * (d->Ci / d->groups), d->Kt * d->Kh * d->Kw, &t)) return "weights too large";
  return "";
}

bool any_active_tap(const Geo& g) {
  // Eq. 4 with unit temporal stride; a general stride is counted directly.
  for (int64_t k = 0; k < g.d.Kt; ++k) {
    if (g.d.stride_t == 1) {
      const int64_t delta = k * g.d.dil_t - g.p_l;
      const int64_t lo = -delta > 0 ? -delta : 0;
      const int64_t hi = g.Z - delta < g.To ? g.Z - delta : g.To;
      if (lo < hi) return true;
    } else {
      for (int64_t t = 0; t < g.To; ++t) {
        const int64_t f = t * g.d.stride_t + k * g.d.dil_t - g.p_l;
        if (f >= 0 && f < g.Z) return true;
      }
    }
  }
  return false;
}

// The two spatial forms of the fast route: 3x3 with stride 1, pad 1,
// dilation 1 (the decoder's main convolutions), and 1x1 with stride 1, pad 0
// (its temporal convolutions, per-frame matrix products).
bool spatial_3x3(const c3c_conv_desc& d) {
  return d.Kh == 3 && d.Kw == 3 && d.stride_h == 1 && d.stride_w == 1 && d.pad_h == 1 &&
         d.pad_w == 1 && d.dil_h == 1 && d.dil_w == 1;
}
bool spatial_1x1(const c3c_conv_desc& d) {
  return d.Kh == 1 && d.Kw == 1 && d.stride_h == 1 && d.stride_w == 1 && d.pad_h == 0 &&
         d.pad_w == 0 && d.dil_h == 1 && d.dil_w == 1;
}

// The route predicate: the first failing clause is the reason.  Temporal
// stride other than 1 is accepted for the 1x1 spatial form only; a single
// temporal tap (Kt = 1) for the 3x3 form only (a per-frame spatial
// convolution), so that a 1x1x1 convolution stays on the fallback.
int decide(const Geo& g, uint32_t mode) {
  const c3c_conv_desc& d = g.d;
  if (mode & C3C_MODE_FORCE_FALLBACK) return C3C_REASON_FORCED;
  if (d.dtype != C3C_DTYPE_BF16 && d.dtype != C3C_DTYPE_F32) return C3C_REASON_DTYPE;
  if (d.groups != 1) return C3C_REASON_GROUPS;
  if (d.stride_t != 1 && !spatial_1x1(d)) return C3C_REASON_STRIDE_T;
  if (d.pad_t_right < 0) return C3C_REASON_PAD_RIGHT;
  if (g.To < 1) return C3C_REASON_NO_OUTPUT;
  if (!any_active_tap(g)) return C3C_REASON_NO_TAP;
  if (d.Kt < 2 && !spatial_3x3(d)) return C3C_REASON_KT1;
  if (!spatial_3x3(d) && !spatial_1x1(d)) return C3C_REASON_SPATIAL;
  return C3C_REASON_NONE;
}

bool overlap(const void* a, int64_t abytes, const void* b, int64_t bbytes) {
  if (!a || !b || abytes <= 0 || bbytes <= 0) return false;
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
  return a0 < b0 + static_cast<uintptr_t>(bbytes) && b0 < a0 + static_cast<uintptr_t>(abytes);
}

int fail(c3c_ctx* ctx, int status, const std::string& msg) {
  if (ctx) ctx->last_error = msg;
  return status;
}

void record_shape(c3c_ctx* ctx, int reason, const c3c_conv_desc& d) {
  for (auto& s : ctx->shapes)
    if (s.reason == reason && std::memcmp(&s.desc, &d, sizeof d) == 0) {
      ++s.count;
      return;
    }
  c3c_sig_count s;
  std::memset(&s, 0, sizeof s);
  s.reason = reason;
  s.desc = d;
  s.count = 1;
  ctx->shapes.push_back(s);
}

}  // namespace
}  // namespace c3c

using namespace c3c;

extern "C" {

int c3c_ctx_create(uint32_t mode, c3c_ctx** out) {
  if (!out || (mode & ~kModeMask)) return C3C_E_INVAL;
  c3c_ctx* c = new (std::nothrow) c3c_ctx();
  if (!c) return C3C_E_INVAL;
  c->mode = mode;
  *out = c;
  return C3C_OK;
}

int c3c_ctx_destroy(c3c_ctx* ctx) {
  delete ctx;
  return C3C_OK;
}

int c3c_set_mode(c3c_ctx* ctx, uint32_t mode) {
  if (!ctx || (mode & ~kModeMask)) return C3C_E_INVAL;
  ctx->mode = mode;
  return C3C_OK;
}

int c3c_get_mode(const c3c_ctx* ctx, uint32_t* mode) {
  if (!ctx || !mode) return C3C_E_INVAL;
  *mode = ctx->mode;
  return C3C_OK;
}

int c3c_output_dims(const c3c_conv_desc* d, int64_t* To, int64_t* Ho, int64_t* Wo, int64_t* L) {
  Geo g;
  if (*make_geo(d, &g)) return C3C_E_INVAL;
  if (To) *To = g.To;
  if (Ho) *Ho = g.Ho;
  if (Wo) *Wo = g.Wo;
  if (L) *L = g.L;
  return C3C_OK;
}

int c3c_tap_interval(const c3c_conv_desc* d, int64_t k, int64_t* o_l, int64_t* o_h) {
  Geo g;
  if (*make_geo(d, &g) || !o_l || !o_h || d->stride_t != 1 || k < 0 || k >= d->Kt)
    return C3C_E_INVAL;
  const int64_t delta = k * d->dil_t - g.p_l;  // Eq. 4
  *o_l = -delta > 0 ? -delta : 0;
  *o_h = g.Z - delta < g.To ? g.Z - delta : g.To;
  return C3C_OK;
}

int c3c_flops(const c3c_conv_desc* d, double* flops) {
  Geo g;
  if (*make_geo(d, &g) || !flops) return C3C_E_INVAL;
  int64_t pairs = 0;
  for (int64_t k = 0; k < d->Kt; ++k) {
    if (d->stride_t == 1) {
      int64_t lo, hi;
      c3c_tap_interval(d, k, &lo, &hi);
      if (hi > lo) pairs += hi - lo;
    } else {
      for (int64_t t = 0; t < g.To; ++t) {
        const int64_t f = t * d->stride_t + k * d->dil_t - g.p_l;
        if (f >= 0 && f < g.Z) ++pairs;
      }
    }
  }
  *flops = 2.0 * double(d->N) * double(d->Co) * double(d->Ci / d->groups) * double(d->Kh) *
           double(d->Kw) * double(g.Ho) * double(g.Wo) * double(pairs);
  return C3C_OK;
}

int c3c_route_query(const c3c_ctx* ctx, const c3c_conv_desc* d, int* route, int* reason) {
  Geo g;
  if (*make_geo(d, &g) || !route || !reason) return C3C_E_INVAL;
  const int r = decide(g, ctx ? ctx->mode : 0u);
  *reason = r;
  *route = r == C3C_REASON_NONE ? C3C_ROUTE_FAST : C3C_ROUTE_FALLBACK;
  return C3C_OK;
}

int c3c_plan_query(const c3c_ctx* ctx, const c3c_conv_desc* d, size_t ws_bytes, c3c_plan* out) {
  Geo g;
  if (*make_geo(d, &g) || !out) return C3C_E_INVAL;
  g.channel_tiles = ctx && (ctx->mode & C3C_MODE_CHANNEL_TILES);
  std::memset(out, 0, sizeof *out);
  const int r = decide(g, ctx ? ctx->mode : 0u);
  out->reason = r;
  out->route = r == C3C_REASON_NONE ? C3C_ROUTE_FAST : C3C_ROUTE_FALLBACK;
  // Stand-in tensor addresses: 256-byte aligned and never dereferenced (a
  // launcher given a LaunchInfo returns before any device call).  Only
  // their alignment and whether they are NULL steer the choices.
  void* const p = reinterpret_cast<void*>(uintptr_t(1) << 20);
  const void* cache = d->Tc > 0 ? p : nullptr;
  void* cache_out = g.L > 0 ? p : nullptr;
  void* ws = ws_bytes > 0 ? p : nullptr;
  LaunchInfo li;
  hipError_t e;
  if (g.To == 0)
    e = hipSuccess;
  else if (r == C3C_REASON_NONE)
    e = launch_fast(g, p, cache, p, p, p, cache_out, ws, static_cast<int64_t>(ws_bytes), nullptr,
                    Fuse{}, &li);
  else
    e = launch_fallback(g, p, cache, p, p, p, nullptr, Fuse{}, &li);
  if (e != hipSuccess && r == C3C_REASON_NONE) {
    // the fast route refuses this size: the call falls back (fast_error)
    out->reason = C3C_REASON_FAST_ERROR;
    out->route = C3C_ROUTE_FALLBACK;
    li = LaunchInfo{};
    e = launch_fallback(g, p, cache, p, p, p, nullptr, Fuse{}, &li);
  }
  if (e != hipSuccess) return C3C_E_INVAL;
  out->kernel = li.kernel;
  out->splits = li.splits;
  out->tile_co = li.tile_co;
  out->tile_h = li.tile_h;
  out->tile_w = li.tile_w;
  out->workgroups = li.workgroups;
  out->cache_in_kernel = li.cache_in_kernel ? 1 : 0;
  return C3C_OK;
}

int c3c_workspace_bytes(const c3c_conv_desc* d, size_t* bytes) {
  Geo g;
  if (*make_geo(d, &g) || !bytes) return C3C_E_INVAL;
  *bytes = 0;
  if (decide(g, 0u) == C3C_REASON_NONE && d->dtype == C3C_DTYPE_BF16 && spatial_3x3(*d))
    *bytes = static_cast<size_t>(fast_bf16_workspace_bytes(g));
  return C3C_OK;
}

namespace {
// the fused form's prologue-pass region: |x| rounded up to 256 bytes, or 0
// when the call would not use one (not bf16, or not the fast 3x3 form)
int64_t prologue_region_bytes(const Geo& g) {
  const c3c_conv_desc& d = g.d;
  if (decide(g, 0u) != C3C_REASON_NONE || d.dtype != C3C_DTYPE_BF16 || !spatial_3x3(d)) return 0;
  const int64_t xb = d.N * d.Ci * d.T * d.H * d.W * 2;
  return (xb + 255) / 256 * 256;
}
}  // namespace

int c3c_fused_workspace_bytes(const c3c_conv_desc* d, size_t* bytes) {
  Geo g;
  if (*make_geo(d, &g) || !bytes) return C3C_E_INVAL;
  const int64_t pr = prologue_region_bytes(g);
  *bytes = pr > 0 ? static_cast<size_t>(pr + fast_bf16_workspace_bytes(g)) : 0;
  return C3C_OK;
}

int c3c_ctx_set_workspace(c3c_ctx* ctx, void* ws, size_t bytes) {
  if (!ctx || (ws == nullptr) != (bytes == 0)) return C3C_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(ws) & 15u) != 0) return C3C_E_INVAL;
  ctx->ws = ws;
  ctx->ws_bytes = bytes;
  return C3C_OK;
}

int c3c_weight_pack_bytes(const c3c_conv_desc* d, size_t* bytes) {
  Geo g;
  if (*make_geo(d, &g) || !bytes) return C3C_E_INVAL;
  if (decide(g, 0u) != C3C_REASON_NONE) {
    *bytes = 0;
    return C3C_OK;
  }
  *bytes = static_cast<size_t>(pack_dims(*d).elems()) * static_cast<size_t>(g.elem);
  return C3C_OK;
}

int c3c_weight_repack(c3c_ctx* ctx, const c3c_conv_desc* d, const void* w, void* wpack,
                      void* stream) {
  Geo g;
  const char* why = make_geo(d, &g);
  if (*why) return fail(ctx, C3C_E_INVAL, why);
  size_t bytes = 0;
  c3c_weight_pack_bytes(d, &bytes);
  if (bytes == 0) return fail(ctx, C3C_E_INVAL, "layer has no fast-route weight layout");
  if (!w || !wpack) return fail(ctx, C3C_E_INVAL, "w and wpack must be non-NULL");
  const int64_t wbytes = d->Co * d->Ci * d->Kt * d->Kh * d->Kw * g.elem;
  if (overlap(w, wbytes, wpack, static_cast<int64_t>(bytes)))
    return fail(ctx, C3C_E_INVAL, "wpack overlaps w");
  const hipError_t e = launch_repack(g, w, wpack, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(ctx, C3C_E_DEVICE, hipGetErrorString(e));
  if (ctx) ++ctx->ctr.repacks;
  return C3C_OK;
}

int c3c_weight_unpack(const c3c_conv_desc* d, const void* wpack, void* w_out, void* stream) {
  Geo g;
  if (*make_geo(d, &g)) return C3C_E_INVAL;
  size_t bytes = 0;
  c3c_weight_pack_bytes(d, &bytes);
  if (bytes == 0 || !wpack || !w_out) return C3C_E_INVAL;
  const int64_t wbytes = d->Co * d->Ci * d->Kt * d->Kh * d->Kw * g.elem;
  if (overlap(w_out, wbytes, wpack, static_cast<int64_t>(bytes))) return C3C_E_INVAL;
  return launch_unpack(g, wpack, w_out, static_cast<hipStream_t>(stream)) == hipSuccess
             ? C3C_OK
             : C3C_E_DEVICE;
}

namespace {

// The normalised block form's pass, run by run_call after every check and
// before the convolution: the new chunk src is normalised and activated into
// the call's x (a region of the workspace).
struct RmsPass {
  const void* src = nullptr;
  const float* gamma = nullptr;
  const float* beta = nullptr;
  float eps = 0.f;
};

// One call, plain or fused (fu: the fused form's prologue / epilogue, or none).
// ws / ws_cap: the split-K (and prologue-pass) workspace: the context's, or
// the library's own scratch for the allocation-free entry point.  pre: the
// block form's normalisation pass (writes x), or none.
int run_call(c3c_ctx* ctx, const c3c_conv_desc* d, const void* x, const void* cache,
             const void* w, const void* wpack, const void* bias, const Fuse& fu, void* y,
             void* cache_out, void* stream, void* ws, size_t ws_cap,
             const RmsPass* pre = nullptr) {
  if (!ctx) return C3C_E_INVAL;
  Geo g;
  const char* why = make_geo(d, &g);
  if (*why) return fail(ctx, C3C_E_INVAL, why);
  g.channel_tiles = (ctx->mode & C3C_MODE_CHANNEL_TILES) != 0;

  // byte extents of every tensor
  const int64_t es = g.elem;
  const int64_t hw = d->H * d->W;
  const int64_t xb = d->N * d->Ci * d->T * hw * es;
  const int64_t cb = d->N * d->Ci * d->Tc * hw * es;
  const int64_t wb = d->Co * (d->Ci / d->groups) * d->Kt * d->Kh * d->Kw * es;
  const int64_t bb = d->has_bias ? d->Co * es : 0;
  const int64_t yb = d->N * d->Co * g.To * g.Ho * g.Wo * es;
  const int64_t ob = d->N * d->Ci * g.L * hw * es;

  if (xb > 0 && !x) return fail(ctx, C3C_E_INVAL, "x is NULL");
  if (cb > 0 && !cache) return fail(ctx, C3C_E_INVAL, "cache is NULL but Tc > 0");
  if (!w) return fail(ctx, C3C_E_INVAL, "w is NULL");
  if (d->has_bias && !bias) return fail(ctx, C3C_E_INVAL, "bias is NULL but has_bias = 1");
  if (yb > 0 && !y) return fail(ctx, C3C_E_INVAL, "y is NULL");
  if (ob > 0 && !cache_out) return fail(ctx, C3C_E_INVAL, "cache_out is NULL but L > 0");
  if (overlap(cache_out, ob, cache, cb) || overlap(cache_out, ob, x, xb))
    return fail(ctx, C3C_E_INVAL, "cache_out overlaps cache or x");
  if (overlap(y, yb, x, xb) || overlap(y, yb, cache, cb) || overlap(y, yb, w, wb) ||
      overlap(y, yb, bias, bb) || overlap(y, yb, cache_out, ob))
    return fail(ctx, C3C_E_INVAL, "y overlaps another tensor");
  const int64_t wsb = static_cast<int64_t>(ws_cap);
  if (overlap(ws, wsb, x, xb) || overlap(ws, wsb, cache, cb) || overlap(ws, wsb, w, wb) ||
      overlap(ws, wsb, bias, bb) || overlap(ws, wsb, y, yb) || overlap(ws, wsb, cache_out, ob))
    return fail(ctx, C3C_E_INVAL, "the context's workspace overlaps a tensor");
  if (fu.any()) {
    if (d->dtype != C3C_DTYPE_BF16) return fail(ctx, C3C_E_INVAL, "the fused form is bf16 only");
    const int64_t sb = fu.pro() ? d->N * d->Ci * 4 : 0;
    const int64_t rb = fu.residual ? yb : 0;
    for (const void* p : {static_cast<const void*>(fu.scale), static_cast<const void*>(fu.shift)})
      if (overlap(p, sb, y, yb) || overlap(p, sb, cache_out, ob) || overlap(p, sb, ws, wsb))
        return fail(ctx, C3C_E_INVAL, "scale or shift overlaps an output");
    if ((fu.residual != y && overlap(fu.residual, rb, y, yb)) || overlap(fu.residual, rb, cache_out, ob) ||
        overlap(fu.residual, rb, ws, wsb))
      return fail(ctx, C3C_E_INVAL, "residual overlaps an output other than y itself");
  }

  const int reason = decide(g, ctx->mode);
  size_t pb = 0;
  if (reason == C3C_REASON_NONE) {
    c3c_weight_pack_bytes(d, &pb);
    if (!wpack) return fail(ctx, C3C_E_INVAL, "wpack is NULL on a call that routes fast");
    if (overlap(y, yb, wpack, static_cast<int64_t>(pb)) ||
        overlap(cache_out, ob, wpack, static_cast<int64_t>(pb)) ||
        overlap(ws, wsb, wpack, static_cast<int64_t>(pb)))
      return fail(ctx, C3C_E_INVAL, "an output or the workspace overlaps wpack");
  }

  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool strict = (ctx->mode & C3C_MODE_STRICT) != 0;
  ++ctx->ctr.calls;

  if (pre) {
    // strict rejections first: the pass runs only for a call that will compute
    if (strict && (reason != C3C_REASON_NONE || (ctx->mode & C3C_MODE_INJECT_FAST_FAILURE))) {
      ++ctx->ctr.strict_rejects;
      return reason != C3C_REASON_NONE
                 ? fail(ctx, C3C_E_UNSUPPORTED, "call does not route fast (strict mode)")
                 : fail(ctx, C3C_E_INJECTED, "injected fast-route failure (strict mode)");
    }
    const hipError_t e = launch_rms_prologue(g, pre->src, pre->gamma, pre->beta, pre->eps,
                                             const_cast<void*>(x), s);
    if (e != hipSuccess) {
      ++ctx->ctr.failed;
      return fail(ctx, C3C_E_DEVICE, hipGetErrorString(e));
    }
  }

  int fb_reason = reason;
  if (reason == C3C_REASON_NONE) {
    hipError_t e = hipSuccess;
    if (ctx->mode & C3C_MODE_INJECT_FAST_FAILURE) {
      if (strict) {
        ++ctx->ctr.strict_rejects;
        return fail(ctx, C3C_E_INJECTED, "injected fast-route failure (strict mode)");
      }
      e = hipErrorLaunchFailure;  // stands for a failure before any launch
    } else {
      // the fused prologue as its own pass when the workspace holds the
      // activated chunk (the 3x3 kernels would evaluate it per staging);
      // the rest of the workspace serves split-K
      const int64_t pr = fu.pro() ? prologue_region_bytes(g) : 0;
      if (pr > 0 && wsb >= pr && d->T > 0) {
        unsigned char* u = static_cast<unsigned char*>(ws);
        e = launch_prologue(g, x, fu.scale, fu.shift, u, s);
        Fuse rest;
        rest.residual = fu.residual;
        if (e == hipSuccess)
          e = launch_fast(g, u, cache, wpack, bias, y, cache_out, u + pr, wsb - pr, s, rest);
      } else {
        e = launch_fast(g, x, cache, wpack, bias, y, cache_out, ws, wsb, s, fu);
      }
    }
    if (e == hipSuccess) {
      ++ctx->ctr.fast;
      return C3C_OK;
    }
    if (strict) {
      ++ctx->ctr.strict_rejects;
      return fail(ctx, C3C_E_DEVICE, hipGetErrorString(e));
    }
    fb_reason = C3C_REASON_FAST_ERROR;
  } else if (strict) {
    ++ctx->ctr.strict_rejects;
    return fail(ctx, C3C_E_UNSUPPORTED, "call does not route fast (strict mode)");
  }
  hipError_t e = launch_fallback(g, x, cache, w, bias, y, s, fu);
  if (e == hipSuccess) e = launch_cache_copy(g, x, cache, cache_out, s, fu);
  if (e != hipSuccess) {
    // nothing was computed: the call counts as failed, not as a fallback
    ++ctx->ctr.failed;
    return fail(ctx, C3C_E_DEVICE, hipGetErrorString(e));
  }
  ++ctx->ctr.fallback;
  if (fb_reason == C3C_REASON_FAST_ERROR)
    ++ctx->ctr.fast_error;
  else if (fb_reason == C3C_REASON_FORCED)
    ++ctx->ctr.forced;
  else
    ++ctx->ctr.unsupported;
  record_shape(ctx, fb_reason, *d);
  return C3C_OK;
}

}  // namespace

int c3c_conv3d_causal_cached(c3c_ctx* ctx, const c3c_conv_desc* d, const void* x,
                             const void* cache, const void* w, const void* wpack,
                             const void* bias, void* y, void* cache_out, void* stream) {
  return run_call(ctx, d, x, cache, w, wpack, bias, Fuse{}, y, cache_out, stream,
                  ctx ? ctx->ws : nullptr, ctx ? ctx->ws_bytes : 0);
}

int c3c_conv3d_causal_cached_noalloc(c3c_ctx* ctx, const c3c_conv_desc* d, const void* x,
                                     const void* cache, const void* w, const void* wpack,
                                     const void* bias, void* y, void* cache_out, void* stream) {
  if (!ctx) return C3C_E_INVAL;
  Geo g;
  const char* why = make_geo(d, &g);
  if (*why) return fail(ctx, C3C_E_INVAL, why);
  // the split-K bytes this call plans for, when it routes fast
  int64_t need = 0;
  if (decide(g, ctx->mode) == C3C_REASON_NONE && d->dtype == C3C_DTYPE_BF16 && spatial_3x3(*d))
    need = fast_bf16_workspace_bytes(g);
  if (need > kNoallocScratchBytes)
    return fail(ctx, C3C_E_INVAL,
                "split-K needs " + std::to_string(need) + " bytes of scratch; the allocation-free "
                "call has " + std::to_string(kNoallocScratchBytes));
  void* ws = nullptr;
  if (need > 0) {
    const hipError_t e = noalloc_scratch(&ws);
    if (e != hipSuccess) return fail(ctx, C3C_E_DEVICE, hipGetErrorString(e));
  }
  return run_call(ctx, d, x, cache, w, wpack, bias, Fuse{}, y, cache_out, stream, ws,
                  static_cast<size_t>(need));
}

int c3c_conv3d_causal_cached_fused(c3c_ctx* ctx, const c3c_conv_desc* d, const void* x,
                                   const void* cache, const void* w, const void* wpack,
                                   const void* bias, const float* scale, const float* shift,
                                   const void* residual, void* y, void* cache_out,
                                   void* stream) {
  if (ctx && (scale == nullptr) != (shift == nullptr))
    return fail(ctx, C3C_E_INVAL, "scale and shift are given together or not at all");
  Fuse fu;
  fu.scale = scale;
  fu.shift = shift;
  fu.residual = static_cast<const uint16_t*>(residual);
  return run_call(ctx, d, x, cache, w, wpack, bias, fu, y, cache_out, stream,
                  ctx ? ctx->ws : nullptr, ctx ? ctx->ws_bytes : 0);
}

int c3c_block_workspace_bytes(const c3c_conv_desc* d, size_t* bytes) {
  Geo g;
  if (*make_geo(d, &g) || !bytes || d->dtype != C3C_DTYPE_BF16) return C3C_E_INVAL;
  const int64_t xb = d->N * d->Ci * d->T * d->H * d->W * 2;
  int64_t splitk = 0;
  if (decide(g, 0u) == C3C_REASON_NONE && spatial_3x3(*d)) splitk = fast_bf16_workspace_bytes(g);
  *bytes = static_cast<size_t>((xb + 255) / 256 * 256 + splitk);
  return C3C_OK;
}

int c3c_conv3d_causal_cached_block(c3c_ctx* ctx, const c3c_conv_desc* d, const void* x,
                                   const void* cache, const void* w, const void* wpack,
                                   const void* bias, const float* gamma, const float* beta,
                                   float eps, const void* residual, void* y, void* cache_out,
                                   void* stream) {
  if (!ctx) return C3C_E_INVAL;
  Geo g;
  const char* why = make_geo(d, &g);
  if (*why) return fail(ctx, C3C_E_INVAL, why);
  if (d->dtype != C3C_DTYPE_BF16) return fail(ctx, C3C_E_INVAL, "the block form is bf16 only");
  if (!gamma || !beta) return fail(ctx, C3C_E_INVAL, "gamma and beta must be non-NULL");
  if (!(eps >= 0.f) || eps > 3.0e38f) return fail(ctx, C3C_E_INVAL, "eps must be finite and >= 0");
  size_t need = 0;
  c3c_block_workspace_bytes(d, &need);
  if (ctx->ws_bytes < need)
    return fail(ctx, C3C_E_INVAL,
                "the block form needs a context workspace of " + std::to_string(need) +
                    " bytes (c3c_block_workspace_bytes); it has " + std::to_string(ctx->ws_bytes));
  const int64_t hw = d->H * d->W;
  const int64_t xb = d->N * d->Ci * d->T * hw * 2;
  const int64_t ub = (xb + 255) / 256 * 256;
  if (xb > 0 && !x) return fail(ctx, C3C_E_INVAL, "x is NULL");
  // the activated chunk takes the workspace's first ub bytes; the rest is the
  // split-K workspace of the convolution that follows
  unsigned char* u = static_cast<unsigned char*>(ctx->ws);
  const int64_t yb = d->N * d->Co * g.To * g.Ho * g.Wo * 2;
  const int64_t ob = d->N * d->Ci * g.L * hw * 2;
  const int64_t gb = d->Ci * 4;
  const int64_t wsb = static_cast<int64_t>(ctx->ws_bytes);
  if (overlap(x, xb, ctx->ws, wsb) || overlap(x, xb, y, yb) || overlap(x, xb, cache_out, ob))
    return fail(ctx, C3C_E_INVAL, "x overlaps an output or the workspace");
  for (const void* p : {static_cast<const void*>(gamma), static_cast<const void*>(beta)})
    if (overlap(p, gb, ctx->ws, wsb) || overlap(p, gb, y, yb) || overlap(p, gb, cache_out, ob))
      return fail(ctx, C3C_E_INVAL, "gamma or beta overlaps an output or the workspace");
  if (overlap(residual, yb, ctx->ws, wsb))
    return fail(ctx, C3C_E_INVAL, "residual overlaps the workspace");
  Fuse fu;
  fu.residual = static_cast<const uint16_t*>(residual);
  RmsPass pre;
  pre.src = x;
  pre.gamma = gamma;
  pre.beta = beta;
  pre.eps = eps;
  return run_call(ctx, d, u, cache, w, wpack, bias, fu, y, cache_out, stream, u + ub,
                  static_cast<size_t>(wsb - ub), &pre);
}

int c3c_counters_get(const c3c_ctx* ctx, c3c_counters* out) {
  if (!ctx || !out) return C3C_E_INVAL;
  *out = ctx->ctr;
  return C3C_OK;
}

int c3c_counters_reset(c3c_ctx* ctx) {
  if (!ctx) return C3C_E_INVAL;
  ctx->ctr = c3c_counters{};
  ctx->shapes.clear();
  return C3C_OK;
}

int c3c_fallback_shapes(const c3c_ctx* ctx, c3c_sig_count* out, int cap, int* n) {
  if (!ctx || !n || cap < 0 || (cap > 0 && !out)) return C3C_E_INVAL;
  const int total = static_cast<int>(ctx->shapes.size());
  for (int i = 0; i < total && i < cap; ++i) out[i] = ctx->shapes[static_cast<size_t>(i)];
  *n = total;
  return C3C_OK;
}

int c3c_mfma_probe(int64_t blocks, int64_t iters, float* out, double* flops, void* stream) {
  if (blocks < 1 || blocks > 0x7fffffff || iters < 1 || iters > 0x7fffffff || !out || !flops)
    return C3C_E_INVAL;
  *flops = mfma_probe_flops(blocks, iters);
  return launch_mfma_probe(blocks, iters, out, static_cast<hipStream_t>(stream)) == hipSuccess
             ? C3C_OK
             : C3C_E_DEVICE;
}

const char* c3c_strerror(int status) {
  switch (status) {
    case C3C_OK: return "ok";
    case C3C_E_INVAL: return "invalid argument";
    case C3C_E_UNSUPPORTED: return "unsupported on the fast route (strict mode)";
    case C3C_E_DEVICE: return "device error";
    case C3C_E_INJECTED: return "injected fast-route failure (strict mode)";
    default: return "unknown status";
  }
}

const char* c3c_last_error(const c3c_ctx* ctx) { return ctx ? ctx->last_error.c_str() : ""; }

}  // extern "C"
