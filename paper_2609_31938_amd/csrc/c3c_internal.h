// Internal interface between the C-ABI host layer (c3c_host.cpp) and the
// kernel translation units.  Not installed; not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "c3c.h"

namespace c3c {

// Geometry of one validated call (Sec. 4.2: |Z|, p_l, T_o; spatial analogue).
struct Geo {
  c3c_conv_desc d;
  int64_t Z;    // |Z|_T = Tc + T
  int64_t p_l;  // effective left pad = pad_t_base - Tc (may be negative)
  int64_t To, Ho, Wo;
  int64_t L;    // new cache length = min(pad_t_base, |Z|)
  int elem;     // bytes per element
  bool channel_tiles = false;  // C3C_MODE_CHANNEL_TILES: no re-tiling of unsplit calls
};

// Fast-route packed-weight layout, in matrix-core fragment order.  One
// fragment covers ROWS output channels and KSTEP input channels of one kernel
// tap (kt, kh, kw); lane l of the wave holds KPL consecutive input channels of
// output channel row l % ROWS:
//   bf16: v_mfma_f32_16x16x32_bf16  ROWS = 16, KSTEP = 32, KPL = 8
//   fp32: v_mfma_f32_32x32x2_f32    ROWS = 32, KSTEP = 2,  KPL = 1
// Element (tap, chunk, cofrag, lane, e) holds
//   w[co = cofrag*ROWS + lane%ROWS][ci = chunk*KSTEP + (lane/ROWS)*KPL + e][tap],
// zero outside [0, Co) x [0, Ci).
struct PackDims {
  int rows;       // output channels per fragment
  int kpl;        // consecutive input channels per lane
  int kstep;      // input channels per fragment = (64 / rows) * kpl
  int64_t taps;   // Kt * Kh * Kw
  int64_t chunks; // ceil(Ci / kstep)
  int64_t cofrags;// ceil(Co / rows)
  int64_t elems() const { return taps * chunks * cofrags * 64 * kpl; }
};
PackDims pack_dims(const c3c_conv_desc& d);

// The fused entry point's optional prologue and epilogue (bf16 calls only).
// scale / shift ([N][Ci] fp32): new-chunk inputs are read as
// RNE_bf16(SiLU(x * scale + shift)), padding stays 0, and frames copied into
// the new cache from the chunk get the same transform.  residual (y's
// layout) is added after the bias, before the one rounding.  Default: none.
struct Fuse {
  const float* scale = nullptr;
  const float* shift = nullptr;
  const uint16_t* residual = nullptr;
  bool pro() const { return scale != nullptr; }
  bool any() const { return scale != nullptr || residual != nullptr; }
};

// What a call would launch, for the plan query (c3c_plan_query): every
// launcher takes an optional LaunchInfo*; when it is given, the launcher
// makes the same choices it makes for a launch, fills it in and returns
// hipSuccess without touching the device.
struct LaunchInfo {
  int kernel = 0;           // enum c3c_kernel
  int64_t tile_co = 0;      // output channels per workgroup
  int64_t tile_h = 0;       // output rows per workgroup (0: a flattened-plane tile)
  int64_t tile_w = 0;       // output columns (or flattened pixels) per workgroup
  int64_t workgroups = 0;   // of the main launch (every split included)
  int splits = 1;
  bool cache_in_kernel = false;
};

hipError_t launch_repack(const Geo& g, const void* w, void* wpack, hipStream_t s);
// measurement support (mfma_probe.hip): back-to-back bf16 matrix-core products
hipError_t launch_mfma_probe(int64_t blocks, int64_t iters, float* out, hipStream_t s);
double mfma_probe_flops(int64_t blocks, int64_t iters);
hipError_t launch_unpack(const Geo& g, const void* wpack, void* w, hipStream_t s);
// ws / ws_bytes: the caller's split-K workspace (may be NULL / 0).
hipError_t launch_fast(const Geo& g, const void* x, const void* cache, const void* wpack,
                       const void* bias, void* y, void* cache_out, void* ws, int64_t ws_bytes,
                       hipStream_t s, const Fuse& fu = Fuse{}, LaunchInfo* info = nullptr);
// bf16 fast kernel (conv_bf16.hip); writes cache_out itself when it can
// (returns *cache_written = true), else the caller copies the cache.  Splits
// the stages of a call too small to fill the device over several workgroups
// when ws holds at least fast_bf16_workspace_bytes(g) bytes (16-byte aligned).
hipError_t launch_fast_bf16(const Geo& g, const void* x, const void* cache, const void* wpack,
                            const void* bias, void* y, void* cache_out, void* ws,
                            int64_t ws_bytes, bool* cache_written, hipStream_t s,
                            const Fuse& fu = Fuse{}, LaunchInfo* info = nullptr);
// fp32 partial-sum bytes a bf16 fast call would split into (0: it runs unsplit)
int64_t fast_bf16_workspace_bytes(const Geo& g);
// fallback, pointwise case (pointwise.hip): 1x1x1, unit spatial stride, no
// spatial padding, one group, bf16 / fp16, aligned buffers
bool pointwise_eligible(const Geo& g, const void* x, const void* cache, const void* w, const void* y);
hipError_t launch_pointwise(const Geo& g, const void* x, const void* cache, const void* w,
                            const void* bias, void* y, hipStream_t s, const Fuse& fu = Fuse{},
                            LaunchInfo* info = nullptr);
// compute units of the current device (256 when no device is visible)
int64_t device_compute_units();
// output channels per workgroup of the two bf16 1x1 kernels of the fast route
constexpr int64_t kTap1x1TileCo = 192;     // conv_tap1x1.hip
constexpr int64_t kPointwiseTileCo = 160;  // pointwise.hip
// fast route, bf16, 1x1 spatial kernel (conv_tap1x1.hip): 192 x 128 output
// tiles on 4 waves (one stage per tap and chunk, or, for one output frame,
// per chunk with all its taps); needs H * W a multiple of 8 and aligned
// pointers.
// tap1x1_blocks is the workgroup count of one output frame per workgroup
// (the routing rule's measure).  Writes the new cache itself when every
// cache frame is among the frames it stages (*cache_written); otherwise the
// caller copies it.
bool tap1x1_eligible(const Geo& g, const void* x, const void* cache, const void* y);
int64_t tap1x1_blocks(const Geo& g);
hipError_t launch_tap1x1(const Geo& g, const void* x, const void* cache, const void* wpack,
                         const void* bias, void* y, void* cache_out, bool* cache_written,
                         hipStream_t s, LaunchInfo* info = nullptr);
// fast route, bf16, 3x3 spatial kernel with Co <= 5 (conv_head.hip): the 9
// spatial taps x Co output channels as the matrix cores' N dimension, then a
// 3x3 gather-sum; needs W a multiple of 8 and aligned pointers.  Writes the
// new cache itself when every cache frame is among the frames it stages
// (*cache_written); otherwise the caller copies it.
bool head_eligible(const Geo& g, const void* x, const void* cache, const void* y);
hipError_t launch_head(const Geo& g, const void* x, const void* cache, const void* wpack,
                       const void* bias, void* y, void* cache_out, bool* cache_written,
                       hipStream_t s, LaunchInfo* info = nullptr);
// fast route, bf16, 1x1 spatial kernel (pointwise.hip): every active temporal
// tap of a call as per-frame matrix products, reading the packed weights; any
// temporal stride and dilation, any H * W and alignment.  The caller copies
// the cache.
hipError_t launch_fast_tap1x1(const Geo& g, const void* x, const void* cache, const void* wpack,
                              const void* bias, void* y, hipStream_t s, const Fuse& fu = Fuse{},
                              LaunchInfo* info = nullptr);
hipError_t launch_fallback(const Geo& g, const void* x, const void* cache, const void* w,
                           const void* bias, void* y, hipStream_t s, const Fuse& fu = Fuse{},
                           LaunchInfo* info = nullptr);
// the fused form's prologue as its own pass: u = RNE_bf16(SiLU(x * scale +
// shift)) over the whole new chunk (fallback.hip)
hipError_t launch_prologue(const Geo& g, const void* x, const float* scale, const float* shift,
                           void* u, hipStream_t s);
hipError_t launch_cache_copy(const Geo& g, const void* x, const void* cache, void* cache_out,
                             hipStream_t s, const Fuse& fu = Fuse{});
// the normalised block form's pass (norm.hip): u = RNE_bf16(SiLU(x * r * gamma
// + beta)), r the per-pixel reciprocal root mean square over the channels
hipError_t launch_rms_prologue(const Geo& g, const void* x, const float* gamma, const float* beta,
                               float eps, void* u, hipStream_t s);
// The allocation-free entry point's split-K scratch (noalloc.hip): a
// file-scope device array of kNoallocScratchBytes; *ptr receives its address
// on the current device (looked up once per device).
constexpr int64_t kNoallocScratchBytes = C3C_NOALLOC_SCRATCH_BYTES;
hipError_t noalloc_scratch(void** ptr);

}  // namespace c3c
