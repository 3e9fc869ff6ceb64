// The normalised block form's prologue as one pass over the new chunk: each
// pixel (n, t, p) of x [N][Ci][T][H*W] (bf16) is normalised by the root mean
// square of its Ci channel values, then a per-channel gain and bias and SiLU
// apply, and one round-to-nearest-even conversion writes u (same layout):
//   r[n,t,p] = 1 / sqrt( (1/Ci) sum_c x[n,c,t,p]^2 + eps )
//   u[n,c,t,p] = RNE_bf16( SiLU( x[n,c,t,p] * r[n,t,p] * gamma[c] + beta[c] ) )
// (the decoder residual block's normalisation and activation ahead of its
// causal convolution; fp32 arithmetic, hardware reciprocal square root,
// exponential and reciprocal).
//
// A workgroup owns 128 consecutive pixels of one (n, t) frame plane and all
// Ci channels.  Vector form (H*W a multiple of 8, 16-byte-aligned x and u):
// thread (channel lane cl = tid / 16, pixel group pg = tid % 16) reads 16-byte
// runs of 8 pixels of channels cl, cl + 16, ...; the 16 channel lanes' partial
// sums of squares meet in LDS, and a second sweep over the same runs (L2-hot)
// writes u; with at most 384 channels the tile stays in registers between
// the two sweeps (all loads in flight at once, x read once).  Scalar form
// otherwise: 128 pixels x 2 channel lanes, 2-byte accesses.  x is read from
// HBM once and u written once: an HBM-bound pass.
#include "c3c_internal.h"
#include "fuse_dev.h"

namespace c3c {
namespace {

constexpr int NPX = 128;  // pixels per workgroup

// Vector form with the whole tile in registers (Ci <= 16 * CPL channel rows,
// CPL per lane): every load of x is issued before the first sum is formed, x
// is read once, and the second sweep works on the registers.  The smallest
// of CPL = 6, 12, 24 that holds the call's channels is launched (fewer
// registers, more workgroups per compute unit).
constexpr int kMaxCpl = 24;
template <int CPL>
__global__ __launch_bounds__(256) void rms_prologue_regs(const uint16_t* __restrict__ x,
                                                         const float* __restrict__ gamma,
                                                         const float* __restrict__ beta, float eps,
                                                         uint16_t* __restrict__ u, int64_t Ci,
                                                         int64_t T, int64_t hw, int64_t tiles) {
  __shared__ float part[16][NPX];
  __shared__ float rr[NPX];
  const int tid = threadIdx.x;
  const int cl = tid >> 4, pg = tid & 15;
  const int64_t b = blockIdx.x;
  const int64_t tile = b % tiles, nt = b / tiles;
  const int64_t n = nt / T, t = nt % T;
  const int64_t p0 = tile * NPX + static_cast<int64_t>(pg) * 8;
  const bool in = p0 < hw;
  const uint16_t* xb = x + ((n * Ci) * T + t) * hw + p0;  // channel 0 of this group
  uint16_t* ub = u + ((n * Ci) * T + t) * hw + p0;
  const int64_t cstride = T * hw;  // elements between channel planes
  fuse_u32x4 v[CPL];
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    const int64_t c = cl + 16 * i;
    v[i] = (in && c < Ci) ? *reinterpret_cast<const fuse_u32x4*>(xb + c * cstride)
                          : fuse_u32x4{0u, 0u, 0u, 0u};
  }
  float ss[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) ss[e] = 0.f;
#pragma unroll
  for (int i = 0; i < CPL; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = fuse_widen(v[i][e] & 0xffffu), hi = fuse_widen(v[i][e] >> 16);
      ss[2 * e] = __builtin_fmaf(lo, lo, ss[2 * e]);
      ss[2 * e + 1] = __builtin_fmaf(hi, hi, ss[2 * e + 1]);
    }
#pragma unroll
  for (int e = 0; e < 8; ++e) part[cl][pg * 8 + e] = ss[e];
  __syncthreads();
  if (tid < NPX) {
    float sum = 0.f;
#pragma unroll
    for (int l = 0; l < 16; ++l) sum += part[l][tid];
    rr[tid] = __builtin_amdgcn_rsqf(sum / static_cast<float>(Ci) + eps);
  }
  __syncthreads();
  if (!in) return;
  float r[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = rr[pg * 8 + e];
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    const int64_t c = cl + 16 * i;
    if (c >= Ci) break;
    const float g = gamma[c], bb = beta[c];
    fuse_u32x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float a = fuse_silu(__builtin_fmaf(fuse_widen(v[i][e] & 0xffffu) * r[2 * e], g, bb));
      const float d = fuse_silu(__builtin_fmaf(fuse_widen(v[i][e] >> 16) * r[2 * e + 1], g, bb));
      o[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector((fuse_f32x2{a, d}), fuse_bf16x2));
    }
    *reinterpret_cast<fuse_u32x4*>(ub + c * cstride) = o;
  }
}

template <bool VEC>
__global__ __launch_bounds__(256) void rms_prologue_pass(const uint16_t* __restrict__ x,
                                                         const float* __restrict__ gamma,
                                                         const float* __restrict__ beta, float eps,
                                                         uint16_t* __restrict__ u, int64_t Ci,
                                                         int64_t T, int64_t hw, int64_t tiles) {
  constexpr int LANES = VEC ? 16 : 2;  // channel lanes
  constexpr int PPT = VEC ? 8 : 1;     // pixels per thread
  __shared__ float part[LANES][NPX];
  __shared__ float rr[NPX];
  const int tid = threadIdx.x;
  const int cl = VEC ? tid >> 4 : tid >> 7;
  const int pg = VEC ? tid & 15 : tid & 127;
  const int64_t b = blockIdx.x;
  const int64_t tile = b % tiles, nt = b / tiles;  // nt = n * T + t
  const int64_t n = nt / T, t = nt % T;
  const int64_t p0 = tile * NPX + static_cast<int64_t>(pg) * PPT;  // this thread's first pixel
  const bool in = p0 < hw;  // VEC: hw % 8 == 0, so a group is all in or all out
  // element (c, p0) of this (n, t) plane
  auto at = [&](int64_t c) { return ((n * Ci + c) * T + t) * hw + p0; };

  float ss[PPT];
#pragma unroll
  for (int e = 0; e < PPT; ++e) ss[e] = 0.f;
  if (in) {
    for (int64_t c = cl; c < Ci; c += LANES) {
      if constexpr (VEC) {
        const fuse_u32x4 v = *reinterpret_cast<const fuse_u32x4*>(x + at(c));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float lo = fuse_widen(v[e] & 0xffffu), hi = fuse_widen(v[e] >> 16);
          ss[2 * e] = __builtin_fmaf(lo, lo, ss[2 * e]);
          ss[2 * e + 1] = __builtin_fmaf(hi, hi, ss[2 * e + 1]);
        }
      } else {
        const float v = fuse_widen(x[at(c)]);
        ss[0] = __builtin_fmaf(v, v, ss[0]);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < PPT; ++e) part[cl][pg * PPT + e] = ss[e];
  __syncthreads();
  if (tid < NPX) {
    float s = 0.f;
#pragma unroll
    for (int l = 0; l < LANES; ++l) s += part[l][tid];
    rr[tid] = __builtin_amdgcn_rsqf(s / static_cast<float>(Ci) + eps);
  }
  __syncthreads();
  if (!in) return;
  float r[PPT];
#pragma unroll
  for (int e = 0; e < PPT; ++e) r[e] = rr[pg * PPT + e];
  for (int64_t c = cl; c < Ci; c += LANES) {
    const float g = gamma[c], bb = beta[c];
    if constexpr (VEC) {
      const fuse_u32x4 v = *reinterpret_cast<const fuse_u32x4*>(x + at(c));
      fuse_u32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float a = fuse_silu(__builtin_fmaf(fuse_widen(v[e] & 0xffffu) * r[2 * e], g, bb));
        const float d = fuse_silu(__builtin_fmaf(fuse_widen(v[e] >> 16) * r[2 * e + 1], g, bb));
        o[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector((fuse_f32x2{a, d}), fuse_bf16x2));
      }
      *reinterpret_cast<fuse_u32x4*>(u + at(c)) = o;
    } else {
      const float a = fuse_silu(__builtin_fmaf(fuse_widen(x[at(c)]) * r[0], g, bb));
      u[at(c)] = static_cast<uint16_t>(
          __builtin_bit_cast(uint32_t, __builtin_convertvector((fuse_f32x2{a, 0.f}), fuse_bf16x2)));
    }
  }
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

hipError_t launch_rms_prologue(const Geo& g, const void* x, const float* gamma, const float* beta,
                               float eps, void* u, hipStream_t s) {
  const c3c_conv_desc& d = g.d;
  const int64_t hw = d.H * d.W;
  if (d.N * d.Ci * d.T * hw == 0) return hipSuccess;
  const int64_t tiles = (hw + NPX - 1) / NPX;
  const int64_t blocks = d.N * d.T * tiles;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  const bool vec = hw % 8 == 0 && aligned16(x) && aligned16(u);
  auto k = !vec                 ? rms_prologue_pass<false>
           : d.Ci <= 16 * 6       ? rms_prologue_regs<6>
           : d.Ci <= 16 * 12      ? rms_prologue_regs<12>
           : d.Ci <= 16 * kMaxCpl ? rms_prologue_regs<kMaxCpl>
                                  : rms_prologue_pass<true>;
  hipLaunchKernelGGL(k, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s,
                     static_cast<const uint16_t*>(x), gamma, beta, eps, static_cast<uint16_t*>(u),
                     d.Ci, d.T, hw, tiles);
  return hipGetLastError();
}

}  // namespace c3c
