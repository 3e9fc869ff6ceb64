// Fallback route: a generic direct Conv3D over the cache-augmented input, and
// the cache-update copy.
//
// The fallback takes every call the fast route does not (the paper returns
// unsupported calls to the original Conv3D, Alg. 1): any kernel size, stride,
// dilation, groups, padding (including a negative effective left pad and a
// right pad), and bf16 / fp16 / fp32 storage, accumulating in fp32.
#include "c3c_internal.h"

#include <hip/hip_fp16.h>

namespace c3c {
namespace {

__device__ inline float load_f(const uint16_t* p, int64_t i, int is_f16) {
  uint16_t v = p[i];
  if (is_f16) return __half2float(__ushort_as_half(v));
  return __uint_as_float(static_cast<uint32_t>(v) << 16);
}
__device__ inline float load_f(const float* p, int64_t i, int) { return p[i]; }

// fp32 -> bf16, round to nearest even; NaN stays NaN.
__device__ inline uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}
__device__ inline void store_f(uint16_t* p, int64_t i, float v, int is_f16) {
  p[i] = is_f16 ? __half_as_ushort(__float2half_rn(v)) : f32_to_bf16(v);
}
__device__ inline void store_f(float* p, int64_t i, float v, int) { p[i] = v; }

struct FbArgs {
  int64_t N, Ci, Co, T, Tc, H, W, Kt, Kh, Kw;
  int64_t st, sh, sw, dt, dh, dw;
  int64_t p_l, ph, pw, groups;
  int64_t Z, To, Ho, Wo;
  int has_bias, is_f16;
};

constexpr int FB_THREADS = 256;

// One thread = one output pixel of one (n, t) frame, for COB output channels
// of one group; the weights it reads are uniform across the block.
template <typename T, int COB>
__global__ __launch_bounds__(FB_THREADS) void fallback_conv3d(FbArgs a, const T* __restrict__ x,
                                                              const T* __restrict__ cache,
                                                              const T* __restrict__ w,
                                                              const T* __restrict__ bias,
                                                              T* __restrict__ y) {
  const int64_t hwo = a.Ho * a.Wo;
  const int64_t p = static_cast<int64_t>(blockIdx.x) * FB_THREADS + threadIdx.x;
  const int64_t cig = a.Ci / a.groups, cog = a.Co / a.groups;
  const int64_t gblocks = (cog + COB - 1) / COB;
  const int64_t g = blockIdx.y / gblocks;
  const int64_t co0 = g * cog + (blockIdx.y % gblocks) * COB;
  const int64_t co_end = min(co0 + COB, (g + 1) * cog);
  const int64_t n = blockIdx.z / a.To, t = blockIdx.z % a.To;
  const bool live = p < hwo;
  const int64_t ho = live ? p / a.Wo : 0, wo = live ? p % a.Wo : 0;
  const int64_t ktaps = a.Kt * a.Kh * a.Kw;
  const int64_t hw = a.H * a.W;

  float acc[COB];
#pragma unroll
  for (int q = 0; q < COB; ++q) acc[q] = 0.f;

  for (int64_t c = 0; c < cig; ++c) {
    const int64_t ci = g * cig + c;
    for (int64_t k = 0; k < a.Kt; ++k) {
      const int64_t tz = t * a.st + k * a.dt - a.p_l;  // Eq. 1 source frame in Z
      if (tz < 0 || tz >= a.Z) continue;
      const T* plane = tz < a.Tc ? cache + ((n * a.Ci + ci) * a.Tc + tz) * hw
                                 : x + ((n * a.Ci + ci) * a.T + (tz - a.Tc)) * hw;
      for (int64_t i = 0; i < a.Kh; ++i) {
        const int64_t hz = ho * a.sh + i * a.dh - a.ph;
        const bool hok = live && hz >= 0 && hz < a.H;
        for (int64_t j = 0; j < a.Kw; ++j) {
          const int64_t wz = wo * a.sw + j * a.dw - a.pw;
          const bool ok = hok && wz >= 0 && wz < a.W;
          const float v = ok ? load_f(plane, hz * a.W + wz, a.is_f16) : 0.f;
          const int64_t widx = (c * a.Kt + k) * a.Kh * a.Kw + i * a.Kw + j;
#pragma unroll
          for (int q = 0; q < COB; ++q) {
            if (co0 + q < co_end) acc[q] += v * load_f(w, (co0 + q) * cig * ktaps + widx, a.is_f16);
          }
        }
      }
    }
  }
  if (!live) return;
#pragma unroll
  for (int q = 0; q < COB; ++q) {
    const int64_t co = co0 + q;
    if (co >= co_end) break;
    float v = acc[q];
    if (a.has_bias) v += load_f(bias, co, a.is_f16);  // bias added once, last
    store_f(y, ((n * a.Co + co) * a.To + t) * hwo + p, v, a.is_f16);
  }
}

template <typename T>
hipError_t launch_fb(const Geo& g, const void* x, const void* cache, const void* w,
                     const void* bias, void* y, hipStream_t s) {
  const c3c_conv_desc& d = g.d;
  FbArgs a;
  a.N = d.N; a.Ci = d.Ci; a.Co = d.Co; a.T = d.T; a.Tc = d.Tc; a.H = d.H; a.W = d.W;
  a.Kt = d.Kt; a.Kh = d.Kh; a.Kw = d.Kw;
  a.st = d.stride_t; a.sh = d.stride_h; a.sw = d.stride_w;
  a.dt = d.dil_t; a.dh = d.dil_h; a.dw = d.dil_w;
  a.p_l = g.p_l; a.ph = d.pad_h; a.pw = d.pad_w; a.groups = d.groups;
  a.Z = g.Z; a.To = g.To; a.Ho = g.Ho; a.Wo = g.Wo;
  a.has_bias = d.has_bias ? 1 : 0;
  a.is_f16 = d.dtype == C3C_DTYPE_F16;
  constexpr int COB = 16;
  const int64_t cog = d.Co / d.groups;
  const int64_t gx = (g.Ho * g.Wo + FB_THREADS - 1) / FB_THREADS;
  const int64_t gy = d.groups * ((cog + COB - 1) / COB);
  const int64_t gz = d.N * g.To;
  if (gx == 0 || gz == 0) return hipSuccess;
  if (gx > 0x7fffffff || gy > 65535 || gz > 65535) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((fallback_conv3d<T, COB>), dim3(gx, gy, gz), dim3(FB_THREADS), 0, s, a,
                     static_cast<const T*>(x), static_cast<const T*>(cache),
                     static_cast<const T*>(w), static_cast<const T*>(bias), static_cast<T*>(y));
  return hipGetLastError();
}

// cache'[n][c][j] = Z[n][c][|Z| - L + j]: whole H*W planes, copied in units
// of U bytes (the largest unit that divides the plane size and the pointers).
template <typename U>
__global__ __launch_bounds__(256) void cache_copy(const U* __restrict__ x, const U* __restrict__ cache,
                                                  U* __restrict__ out, int64_t planes, int64_t units,
                                                  int64_t Ci, int64_t L, int64_t T, int64_t Tc,
                                                  int64_t Z) {
  for (int64_t pl = blockIdx.y; pl < planes; pl += gridDim.y) {
    const int64_t j = pl % L, nc = pl / L;  // nc = n * Ci + c
    const int64_t f = Z - L + j;
    const U* src = f < Tc ? cache + (nc * Tc + f) * units : x + (nc * T + (f - Tc)) * units;
    U* dst = out + pl * units;
    for (int64_t u = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; u < units;
         u += static_cast<int64_t>(gridDim.x) * 256)
      dst[u] = src[u];
  }
  (void)Ci;
}

template <typename U>
hipError_t launch_cc(const Geo& g, const void* x, const void* cache, void* out, hipStream_t s) {
  const c3c_conv_desc& d = g.d;
  const int64_t plane_bytes = d.H * d.W * g.elem;
  const int64_t units = plane_bytes / static_cast<int64_t>(sizeof(U));
  const int64_t planes = d.N * d.Ci * g.L;
  int64_t gx = (units + 255) / 256;
  if (gx > 4096) gx = 4096;
  const int64_t gy = planes < 65535 ? planes : 65535;
  hipLaunchKernelGGL((cache_copy<U>), dim3(gx, gy), dim3(256), 0, s, static_cast<const U*>(x),
                     static_cast<const U*>(cache), static_cast<U*>(out), planes, units, d.Ci, g.L,
                     d.T, d.Tc, g.Z);
  return hipGetLastError();
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

}  // namespace

hipError_t launch_fallback(const Geo& g, const void* x, const void* cache, const void* w,
                           const void* bias, void* y, hipStream_t s) {
  if (g.To == 0) return hipSuccess;
  if (g.d.dtype == C3C_DTYPE_F32) return launch_fb<float>(g, x, cache, w, bias, y, s);
  return launch_fb<uint16_t>(g, x, cache, w, bias, y, s);
}

hipError_t launch_cache_copy(const Geo& g, const void* x, const void* cache, void* cache_out,
                             hipStream_t s) {
  if (g.L == 0) return hipSuccess;
  const int64_t plane_bytes = g.d.H * g.d.W * g.elem;
  auto fits = [&](size_t a) {
    return plane_bytes % static_cast<int64_t>(a) == 0 && aligned(cache_out, a) &&
           (x == nullptr || aligned(x, a)) && (cache == nullptr || aligned(cache, a));
  };
  if (fits(16)) return launch_cc<uint4>(g, x, cache, cache_out, s);
  if (fits(4)) return launch_cc<uint32_t>(g, x, cache, cache_out, s);
  return launch_cc<uint16_t>(g, x, cache, cache_out, s);
}

}  // namespace c3c
