// Fallback route: a generic direct Conv3D over the cache-augmented input, and
// the cache-update copy.
//
// The fallback takes every call the fast route does not (the paper returns
// unsupported calls to the original Conv3D, Alg. 1): any kernel size, stride,
// dilation, groups, padding (including a negative effective left pad and a
// right pad), and bf16 / fp16 / fp32 storage, accumulating in fp32.  Pointwise
// (1x1x1) bf16 / fp16 calls go to the matrix-core kernel in pointwise.hip.
#include "c3c_internal.h"
#include "fuse_dev.h"

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
  // the fused form (bf16 only; NULL when absent): the prologue's per-(n, ci)
  // scale and shift, applied to the new chunk's in-range values, and the
  // residual added after the bias
  const float* scale;
  const float* shift;
  const uint16_t* residual;
};

constexpr int FB_THREADS = 256;
constexpr int FB_PPT = 2;                         // output pixels per thread
constexpr int FB_COB = 32;                        // output channels per workgroup
constexpr int FB_WROW = FB_COB + 4;               // LDS floats per staged pair (padded)
constexpr int FB_PAIRS = 224;                     // (input channel, tap) pairs per chunk
constexpr int FB_U = 8;                           // pairs whose loads are in flight together

template <typename T>
struct Buf;
template <>
struct Buf<uint16_t> {
  static __device__ inline float load(__amdgpu_buffer_rsrc_t r, uint32_t off, int is_f16) {
    const uint16_t v = __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
    return is_f16 ? __half2float(__ushort_as_half(v)) : __uint_as_float(static_cast<uint32_t>(v) << 16);
  }
};
template <>
struct Buf<float> {
  static __device__ inline float load(__amdgpu_buffer_rsrc_t r, uint32_t off, int) {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
  }
};

// Workgroup = FB_THREADS * FB_PPT consecutive output pixels of one (n, t)
// frame x FB_COB output channels of one group.  The weights of a chunk of
// (input channel, tap) pairs for the FB_COB output channels are staged in
// LDS as fp32 [pair][co]; every lane of a wave reads the same weight address
// (a broadcast), so each input value a thread loads feeds FB_COB fp32 FMAs.
// Input values are read through a buffer resource per source frame plane:
// padding positions (and frames outside Z) are out-of-range offsets that
// load as zero, so the loop has no branches and the loads of FB_U pairs are
// in flight together.
template <typename T>
__global__ __launch_bounds__(FB_THREADS) void fallback_conv3d(FbArgs a, const T* __restrict__ x,
                                                              const T* __restrict__ cache,
                                                              const T* __restrict__ w,
                                                              const T* __restrict__ bias,
                                                              T* __restrict__ y) {
  __shared__ __align__(16) float wl[FB_PAIRS * FB_WROW];
  constexpr uint32_t OOB = 0x80000000u;
  const int64_t hwo = a.Ho * a.Wo;
  const int64_t cig = a.Ci / a.groups, cog = a.Co / a.groups;
  const int64_t gblocks = (cog + FB_COB - 1) / FB_COB;
  const int64_t g = blockIdx.y / gblocks;
  const int64_t co0 = g * cog + (blockIdx.y % gblocks) * FB_COB;
  const int ncob = static_cast<int>(min(static_cast<int64_t>(FB_COB), (g + 1) * cog - co0));
  const int64_t n = blockIdx.z / a.To, t = blockIdx.z % a.To;
  const int64_t taps = a.Kt * a.Kh * a.Kw;
  const int64_t hw = a.H * a.W;
  const int64_t npairs = cig * taps;
  const int esz = static_cast<int>(sizeof(T));
  const int plane_bytes = static_cast<int>(hw * esz);

  // per-pixel spatial origin of the receptive field (a plane is < 2^31 bytes)
  int hb[FB_PPT], wb[FB_PPT];
  bool live[FB_PPT];
  int64_t pix[FB_PPT];
#pragma unroll
  for (int q = 0; q < FB_PPT; ++q) {
    const int64_t p = static_cast<int64_t>(blockIdx.x) * FB_THREADS * FB_PPT + q * FB_THREADS + threadIdx.x;
    live[q] = p < hwo;
    pix[q] = p;
    const int pp = live[q] ? static_cast<int>(p) : 0;
    const int wo = static_cast<int>(a.Wo);
    hb[q] = (pp / wo) * static_cast<int>(a.sh) - static_cast<int>(a.ph);
    wb[q] = (pp % wo) * static_cast<int>(a.sw) - static_cast<int>(a.pw);
  }
  float acc[FB_PPT][FB_COB];
#pragma unroll
  for (int q = 0; q < FB_PPT; ++q)
#pragma unroll
    for (int c = 0; c < FB_COB; ++c) acc[q][c] = 0.f;

  const int Kt = static_cast<int>(a.Kt), Kh = static_cast<int>(a.Kh), Kw = static_cast<int>(a.Kw);
  const int H = static_cast<int>(a.H), W = static_cast<int>(a.W);
  const int dh = static_cast<int>(a.dh), dw = static_cast<int>(a.dw);
  for (int64_t r0 = 0; r0 < npairs; r0 += FB_PAIRS) {
    const int np = static_cast<int>(min(static_cast<int64_t>(FB_PAIRS), npairs - r0));
    __syncthreads();
    // stage w[co0 + co][pair r0 + r] -> wl[r * FB_WROW + co], pairs contiguous
    // in global memory (pair = ci * taps + tap), so consecutive threads read
    // consecutive pairs
    for (int e = threadIdx.x; e < np * FB_COB; e += FB_THREADS) {
      const int r = e % np, co = e / np;
      wl[r * FB_WROW + co] = co < ncob ? load_f(w, (co0 + co) * npairs + r0 + r, a.is_f16) : 0.f;
    }
    __syncthreads();
    // wave-uniform (ci, k, i, j) of the chunk's first pair, then advanced in order
    int ci = static_cast<int>(r0 / taps);
    int tap = static_cast<int>(r0 % taps);
    int k = tap / (Kh * Kw), i = (tap / Kw) % Kh, j = tap % Kw;
    for (int r = 0; r < np; r += FB_U) {
      float v[FB_U][FB_PPT];
#pragma unroll
      for (int u = 0; u < FB_U; ++u) {
        const int64_t tz = t * a.st + k * a.dt - a.p_l;  // Eq. 1 source frame in Z
        const bool fok = (r + u < np) & (tz >= 0) & (tz < a.Z);
        const int64_t cin = g * cig + ci;
        const T* plane = !fok ? x : tz < a.Tc ? cache + ((n * a.Ci + cin) * a.Tc + tz) * hw
                                              : x + ((n * a.Ci + cin) * a.T + (tz - a.Tc)) * hw;
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<T*>(plane), 0, fok ? plane_bytes : 0, 0x00020000);
        // fused prologue on values of the new chunk (tz >= Tc); padding stays 0
        const bool pro = a.scale != nullptr && fok && tz >= a.Tc;
        const float psc = pro ? a.scale[n * a.Ci + cin] : 0.f, psh = pro ? a.shift[n * a.Ci + cin] : 0.f;
#pragma unroll
        for (int q = 0; q < FB_PPT; ++q) {
          const int hz = hb[q] + i * dh, wz = wb[q] + j * dw;
          const bool ok = live[q] & (hz >= 0) & (hz < H) & (wz >= 0) & (wz < W);
          v[u][q] = Buf<T>::load(rs, ok ? static_cast<uint32_t>((hz * W + wz) * esz) : OOB, a.is_f16);
          if (pro && ok) v[u][q] = fuse_value(v[u][q], psc, psh);
        }
        if (++j == Kw) {
          j = 0;
          if (++i == Kh) {
            i = 0;
            if (++k == Kt) {
              k = 0;
              ++ci;
            }
          }
        }
      }
      // guards, never `break`: an early exit would make the accumulator
      // indices dynamic and push the accumulators to scratch memory
#pragma unroll
      for (int u = 0; u < FB_U; ++u) {
        if (r + u >= np) continue;
        const float4* wv = reinterpret_cast<const float4*>(wl + (r + u) * FB_WROW);
#pragma unroll
        for (int c4 = 0; c4 < FB_COB / 4; ++c4) {
          const float4 ww = wv[c4];
#pragma unroll
          for (int q = 0; q < FB_PPT; ++q) {
            acc[q][4 * c4 + 0] += v[u][q] * ww.x;
            acc[q][4 * c4 + 1] += v[u][q] * ww.y;
            acc[q][4 * c4 + 2] += v[u][q] * ww.z;
            acc[q][4 * c4 + 3] += v[u][q] * ww.w;
          }
        }
      }
    }
  }
#pragma unroll
  for (int q = 0; q < FB_PPT; ++q) {
    if (!live[q]) continue;
    const int64_t p = pix[q];
#pragma unroll
    for (int c = 0; c < FB_COB; ++c) {
      if (c >= ncob) continue;
      const int64_t co = co0 + c;
      float v = acc[q][c];
      if (a.has_bias) v += load_f(bias, co, a.is_f16);  // bias added once, last
      const int64_t yi = ((n * a.Co + co) * a.To + t) * hwo + p;
      if (a.residual) v += fuse_widen(a.residual[yi]);  // fused residual, before the rounding
      store_f(y, yi, v, a.is_f16);
    }
  }
}

template <typename T>
hipError_t launch_fb(const Geo& g, const void* x, const void* cache, const void* w,
                     const void* bias, void* y, hipStream_t s, const Fuse& fu, LaunchInfo* info) {
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
  a.scale = fu.scale;
  a.shift = fu.shift;
  a.residual = fu.residual;
  const int64_t cog = d.Co / d.groups;
  const int64_t gx = (g.Ho * g.Wo + FB_THREADS * FB_PPT - 1) / (FB_THREADS * FB_PPT);
  const int64_t gy = d.groups * ((cog + FB_COB - 1) / FB_COB);
  const int64_t gz = d.N * g.To;
  if (info) {
    info->kernel = C3C_KERNEL_FALLBACK_DIRECT;
    info->tile_co = FB_COB;
    info->tile_h = 0;
    info->tile_w = FB_THREADS * FB_PPT;
    info->workgroups = gx * gy * gz;
    return hipSuccess;
  }
  if (gx == 0 || gz == 0) return hipSuccess;
  if (gx > 0x7fffffff || gy > 65535 || gz > 65535) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((fallback_conv3d<T>), dim3(gx, gy, gz), dim3(FB_THREADS), 0, s, a,
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

// The same copy for the fused form: planes that come from the new chunk get
// the prologue (bf16), planes from the old cache are copied as they are.
// VEC: 8 elements per step (16-byte units), else one.
template <bool VEC>
__global__ __launch_bounds__(256) void cache_copy_pro(const uint16_t* __restrict__ x,
                                                      const uint16_t* __restrict__ cache,
                                                      uint16_t* __restrict__ out,
                                                      const float* __restrict__ scale,
                                                      const float* __restrict__ shift, int64_t planes,
                                                      int64_t hw, int64_t L, int64_t T, int64_t Tc,
                                                      int64_t Z) {
  const int64_t units = VEC ? hw / 8 : hw;
  for (int64_t pl = blockIdx.y; pl < planes; pl += gridDim.y) {
    const int64_t j = pl % L, nc = pl / L;  // nc = n * Ci + c
    const int64_t f = Z - L + j;
    const bool from_x = f >= Tc;
    const uint16_t* src = from_x ? x + (nc * T + (f - Tc)) * hw : cache + (nc * Tc + f) * hw;
    const float s = from_x ? scale[nc] : 0.f, t = from_x ? shift[nc] : 0.f;
    uint16_t* dst = out + pl * hw;
    for (int64_t u = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; u < units;
         u += static_cast<int64_t>(gridDim.x) * 256) {
      if (VEC) {
        const fuse_u32x4 v = reinterpret_cast<const fuse_u32x4*>(src)[u];
        reinterpret_cast<fuse_u32x4*>(dst)[u] = from_x ? fuse_seg8(v, s, t, true) : v;
      } else {
        const uint16_t v = src[u];
        dst[u] = from_x ? fuse_one(v, s, t, true) : v;
      }
    }
  }
}

// The fused form's prologue as a pass of its own over the new chunk
// [N * Ci rows][T * H * W]: u = RNE_bf16(SiLU(x * scale[row] + shift[row])).
// VEC: 8 elements per step (16-byte units).
template <bool VEC>
__global__ __launch_bounds__(256) void prologue_pass(const uint16_t* __restrict__ x,
                                                     const float* __restrict__ scale,
                                                     const float* __restrict__ shift,
                                                     uint16_t* __restrict__ u, int64_t rows,
                                                     int64_t row_len) {
  const int64_t units = VEC ? row_len / 8 : row_len;
  for (int64_t r = blockIdx.y; r < rows; r += gridDim.y) {
    const float s = scale[r], t = shift[r];
    const uint16_t* src = x + r * row_len;
    uint16_t* dst = u + r * row_len;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < units;
         i += static_cast<int64_t>(gridDim.x) * 256) {
      if (VEC)
        reinterpret_cast<fuse_u32x4*>(dst)[i] = fuse_seg8(reinterpret_cast<const fuse_u32x4*>(src)[i], s, t, true);
      else
        dst[i] = fuse_one(src[i], s, t, true);
    }
  }
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

}  // namespace

hipError_t launch_fallback(const Geo& g, const void* x, const void* cache, const void* w,
                           const void* bias, void* y, hipStream_t s, const Fuse& fu,
                           LaunchInfo* info) {
  if (g.To == 0) return hipSuccess;
  // the pointwise kernel's aligned epilogue also reads the residual 8 bytes at a time
  if (pointwise_eligible(g, x, cache, w, y) &&
      (fu.residual == nullptr || (reinterpret_cast<uintptr_t>(fu.residual) & 7) == 0))
    return launch_pointwise(g, x, cache, w, bias, y, s, fu, info);
  if (g.d.dtype == C3C_DTYPE_F32) return launch_fb<float>(g, x, cache, w, bias, y, s, fu, info);
  return launch_fb<uint16_t>(g, x, cache, w, bias, y, s, fu, info);
}

hipError_t launch_prologue(const Geo& g, const void* x, const float* scale, const float* shift,
                           void* u, hipStream_t s) {
  const c3c_conv_desc& d = g.d;
  const int64_t rows = d.N * d.Ci, row_len = d.T * d.H * d.W;
  if (rows == 0 || row_len == 0) return hipSuccess;
  const bool vec = row_len % 8 == 0 && aligned(x, 16) && aligned(u, 16);
  int64_t gx = ((vec ? row_len / 8 : row_len) + 255) / 256;
  if (gx > 4096) gx = 4096;
  const int64_t gy = rows < 65535 ? rows : 65535;
  auto k = vec ? prologue_pass<true> : prologue_pass<false>;
  hipLaunchKernelGGL(k, dim3(gx, gy), dim3(256), 0, s, static_cast<const uint16_t*>(x), scale, shift,
                     static_cast<uint16_t*>(u), rows, row_len);
  return hipGetLastError();
}

hipError_t launch_cache_copy(const Geo& g, const void* x, const void* cache, void* cache_out,
                             hipStream_t s, const Fuse& fu) {
  if (g.L == 0) return hipSuccess;
  if (fu.pro() && g.d.T > 0) {
    const c3c_conv_desc& d = g.d;
    const int64_t hw = d.H * d.W, planes = d.N * d.Ci * g.L;
    const bool vec = hw % 8 == 0 && aligned(cache_out, 16) && aligned(x, 16) &&
                     (cache == nullptr || aligned(cache, 16));
    int64_t gx = ((vec ? hw / 8 : hw) + 255) / 256;
    if (gx > 4096) gx = 4096;
    const int64_t gy = planes < 65535 ? planes : 65535;
    auto k = vec ? cache_copy_pro<true> : cache_copy_pro<false>;
    hipLaunchKernelGGL(k, dim3(gx, gy), dim3(256), 0, s, static_cast<const uint16_t*>(x),
                       static_cast<const uint16_t*>(cache), static_cast<uint16_t*>(cache_out),
                       fu.scale, fu.shift, planes, hw, g.L, d.T, d.Tc, g.Z);
    return hipGetLastError();
  }
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
