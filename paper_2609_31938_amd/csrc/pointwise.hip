// Fallback route, pointwise case.  A 1x1x1 Conv3D (stride 1 and no padding in
// H and W, one group) reads a single temporal tap: output frame t is, for each
// batch element, the matrix product y[co][p] = sum_ci w[co][ci] z[ci][p] over
// the pixels p of source frame f = t * s_t - p_l of [cache; x] (zero when f is
// outside it), plus the bias once (the cached-conv definition, Eq. 1-2, with
// Kt = Kh = Kw = 1).  bf16 / fp16 storage, matrix cores, fp32 accumulation.
//
// Workgroup = 160 output channels x 128 consecutive pixels of one (n, t)
// frame; four waves of 80 channels x 64 pixels.  Per 32-channel chunk the
// activation tile [32 ch][128 px] is copied into LDS as it lies in memory
// (pixels contiguous, as NCTHW stores them), and the transposing LDS read
// ds_read_b64_tr_b16 turns it into the matrix-core operand (8 consecutive
// channels of one pixel per lane).  Weights come straight from the unpacked
// w[co][ci] rows (8 consecutive channels of one output channel per lane).
#include "c3c_internal.h"

namespace c3c {
namespace {

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int PW_K = 32;       // input channels per chunk (one matrix-core K step)
constexpr int PW_PX = 128;     // pixels per workgroup
constexpr int PW_WCO = 5;      // 16-channel output fragments per wave
constexpr int PW_NPF = 4;      // 16-pixel fragments per wave
constexpr int PW_CO = 2 * 16 * PW_WCO;  // output channels per workgroup
// LDS bytes per staged channel row: 128 px * 2 B + 32 B.  The pad makes the
// row stride 8 banks mod 64, so the 4 channel rows x 4 pixel groups that one
// 16-lane block of a transposing read touches fall in distinct banks.
constexpr int PW_PITCH = PW_PX * 2 + 32;
constexpr int PW_BUF = PW_K * PW_PITCH;

struct PwArgs {
  const uint16_t* x;
  const uint16_t* cache;
  const uint16_t* w;
  const uint16_t* bias;
  uint16_t* y;
  int64_t hw;
  int N, Ci, Co, T, Tc, To, Z, st, p_l;
  int chunks, px_tiles, co_tiles;
  int has_bias;
};

__device__ inline uint16_t to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}
__device__ inline uint16_t to_f16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<_Float16>(f));
}
__device__ inline float from_b16(uint16_t v, bool f16) {
  return f16 ? static_cast<float>(__builtin_bit_cast(_Float16, v))
             : __uint_as_float(static_cast<uint32_t>(v) << 16);
}

template <bool F16>
__device__ inline f32x4 mma(i16x8 a, u32x4 b, f32x4 c) {
  if constexpr (F16)
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

template <bool F16>
__global__ __launch_bounds__(256) void pointwise_conv(PwArgs a) {
  __shared__ __align__(16) unsigned char lds[2 * PW_BUF];
  constexpr uint32_t OOB = 0x80000000u;  // beyond every resource's size
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wco = wave & 1, wpx = wave >> 1;

  int b = blockIdx.x;
  const int pt = b % a.px_tiles;
  b /= a.px_tiles;
  const int ctile = b % a.co_tiles;
  b /= a.co_tiles;
  const int t = b % a.To;
  const int n = b / a.To;
  const int px0 = pt * PW_PX;
  const int f = t * a.st - a.p_l;
  const bool fok = f >= 0 && f < a.Z;

  // source frame plane of channel 0 (pixel px0) and the channel-plane stride
  const uint16_t* src;
  int64_t cstride;
  if (f < a.Tc) {
    cstride = static_cast<int64_t>(a.Tc) * a.hw;
    src = a.cache + static_cast<int64_t>(n) * a.Ci * cstride + static_cast<int64_t>(f) * a.hw + px0;
  } else {
    cstride = static_cast<int64_t>(a.T) * a.hw;
    src = a.x + static_cast<int64_t>(n) * a.Ci * cstride + static_cast<int64_t>(f - a.Tc) * a.hw + px0;
  }
  const uint32_t cs = static_cast<uint32_t>(cstride * 2);
  // chunk c's resource starts at channel 32c and ends after the last real
  // channel's row of this frame: channels past Ci load as 0; a frame outside
  // Z has an empty resource (the output is the bias alone)
  auto chunk_rsrc = [&](int c) {
    const int c0 = c * PW_K;
    int64_t bytes = ((a.Ci - 1 - c0) * cstride + a.hw - px0) * 2;
    if (!fok || bytes < 0) bytes = 0;
    if (bytes > 0x7fffffff) bytes = 0x7fffffff;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(src + (fok ? c0 * cstride : 0)), 0,
                                             static_cast<int>(bytes), 0x00020000);
  };

  // staging: thread -> channel row tid / 8, pixels 16 * (tid % 8) .. + 15
  const int sch = tid >> 3, spx = (tid & 7) * 16;
  const uint32_t soff = static_cast<uint32_t>(sch) * cs + static_cast<uint32_t>(spx) * 2u;
  const int slds = sch * PW_PITCH + spx * 2;
  u32x4 sv[2];
  auto load_chunk = [&](int c) {
    const __amdgpu_buffer_rsrc_t rs = chunk_rsrc(c);
    sv[0] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, soff, 0, 0));
    sv[1] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, soff + 16u, 0, 0));
  };
  auto store_chunk = [&](int buf) {
    *reinterpret_cast<u32x4*>(lds + buf * PW_BUF + slds) = sv[0];
    *reinterpret_cast<u32x4*>(lds + buf * PW_BUF + slds + 16) = sv[1];
  };

  // weights: lane l holds w[co = frag * 16 + l % 16][ci = 32c + 8 (l / 16) .. + 7];
  // rows past Co and channels past Ci are out-of-range offsets (zeros)
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.w), 0, static_cast<int>(static_cast<int64_t>(a.Co) * a.Ci * 2), 0x00020000);
  const int cof0 = ctile * PW_CO + wco * 16 * PW_WCO + (lane & 15);
  const int wci = 8 * (lane >> 4);
  u32x4 wv[PW_WCO];
  auto load_w = [&](int c) {
    const int ci = c * PW_K + wci;
#pragma unroll
    for (int cf = 0; cf < PW_WCO; ++cf) {
      const int co = cof0 + 16 * cf;
      const uint32_t off = (co < a.Co) & (ci < a.Ci)
                               ? static_cast<uint32_t>(co * a.Ci + ci) * 2u : OOB;
      wv[cf] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(wrs, off, 0, 0));
    }
  };

  // transposing operand read: within each 16-lane block (channel group
  // g = l / 16), lane j names channel 8g + 4h + j / 4 at pixel group
  // 4 (j % 4) of the fragment; lane j receives channels 8g + 4h .. + 3 of
  // the fragment's pixel j
  const int j = lane & 15, g = lane >> 4;
  const int ra = (8 * g + (j >> 2)) * PW_PITCH + (wpx * 16 * PW_NPF + 4 * (j & 3)) * 2;
  auto read_a = [&](int buf, int pf) {
    const unsigned char* p = lds + buf * PW_BUF + ra + pf * 32;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 4 * PW_PITCH));
    return i16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  };

  f32x4 acc[PW_WCO][PW_NPF];
#pragma unroll
  for (int cf = 0; cf < PW_WCO; ++cf)
#pragma unroll
    for (int pf = 0; pf < PW_NPF; ++pf) acc[cf][pf] = f32x4{0.f, 0.f, 0.f, 0.f};

  load_chunk(0);
  store_chunk(0);
  __syncthreads();
  for (int c = 0; c < a.chunks; ++c) {
    const int buf = c & 1;
    if (c + 1 < a.chunks) load_chunk(c + 1);
    load_w(c);
    i16x8 av[PW_NPF];
#pragma unroll
    for (int pf = 0; pf < PW_NPF; ++pf) av[pf] = read_a(buf, pf);
#pragma unroll
    for (int pf = 0; pf < PW_NPF; ++pf)
#pragma unroll
      for (int cf = 0; cf < PW_WCO; ++cf) acc[cf][pf] = mma<F16>(av[pf], wv[cf], acc[cf][pf]);
    // the other buffer was last read in chunk c - 1, before the barrier that
    // ended it
    if (c + 1 < a.chunks) store_chunk(buf ^ 1);
    __syncthreads();
  }

  // epilogue: lane l holds pixels 4 (l / 16) .. + 3 of output channel l % 16
  // of each fragment; bias once, one rounding, NCTHW store
  uint16_t* ybase = a.y + (static_cast<int64_t>(n) * a.Co * a.To + t) * a.hw;
#pragma unroll
  for (int cf = 0; cf < PW_WCO; ++cf) {
    const int co = cof0 + 16 * cf;
    if (co >= a.Co) continue;
    const float bb = a.has_bias ? from_b16(a.bias[co], F16) : 0.f;
    uint16_t* yrow = ybase + static_cast<int64_t>(co) * a.To * a.hw;
#pragma unroll
    for (int pf = 0; pf < PW_NPF; ++pf) {
      const int p = px0 + wpx * 16 * PW_NPF + pf * 16 + 4 * g;
      uint16_t v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = F16 ? to_f16(acc[cf][pf][r] + bb) : to_bf16(acc[cf][pf][r] + bb);
      if (p + 4 <= a.hw) {
        *reinterpret_cast<uint2*>(yrow + p) = make_uint2(v[0] | (static_cast<uint32_t>(v[1]) << 16),
                                                        v[2] | (static_cast<uint32_t>(v[3]) << 16));
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (p + r < a.hw) yrow[p + r] = v[r];
      }
    }
  }
}

bool aligned(const void* p, uintptr_t m) { return (reinterpret_cast<uintptr_t>(p) & (m - 1)) == 0; }

}  // namespace

bool pointwise_eligible(const Geo& g, const void* x, const void* cache, const void* w, const void* y) {
  const c3c_conv_desc& d = g.d;
  if (d.dtype != C3C_DTYPE_BF16 && d.dtype != C3C_DTYPE_F16) return false;
  if (d.Kt != 1 || d.Kh != 1 || d.Kw != 1 || d.groups != 1) return false;
  if (d.stride_h != 1 || d.stride_w != 1 || d.pad_h != 0 || d.pad_w != 0) return false;
  const int64_t hw = d.H * d.W;
  // 16-byte loads of 8 pixels / 8 channels and 8-byte stores of 4 pixels
  if (hw % 8 != 0 || d.Ci % 8 != 0) return false;
  if (!aligned(x, 16) || (cache != nullptr && !aligned(cache, 16)) || !aligned(w, 16) || !aligned(y, 8))
    return false;
  // 32-bit buffer offsets: one 32-channel chunk of a source frame and the
  // weights must each span less than 2 GiB
  const int64_t frames = d.T > d.Tc ? d.T : d.Tc;
  if (static_cast<int64_t>(PW_K) * frames * hw * 2 >= 0x7fffffff) return false;
  if (d.Co * d.Ci * 2 >= 0x7fffffff) return false;
  return true;
}

hipError_t launch_pointwise(const Geo& g, const void* x, const void* cache, const void* w,
                            const void* bias, void* y, hipStream_t s) {
  const c3c_conv_desc& d = g.d;
  PwArgs a;
  a.x = static_cast<const uint16_t*>(x);
  a.cache = static_cast<const uint16_t*>(cache);
  a.w = static_cast<const uint16_t*>(w);
  a.bias = static_cast<const uint16_t*>(bias);
  a.y = static_cast<uint16_t*>(y);
  a.hw = d.H * d.W;
  a.N = static_cast<int>(d.N);
  a.Ci = static_cast<int>(d.Ci);
  a.Co = static_cast<int>(d.Co);
  a.T = static_cast<int>(d.T);
  a.Tc = static_cast<int>(d.Tc);
  a.To = static_cast<int>(g.To);
  a.Z = static_cast<int>(g.Z);
  a.st = static_cast<int>(d.stride_t);
  a.p_l = static_cast<int>(g.p_l);
  a.chunks = static_cast<int>((d.Ci + PW_K - 1) / PW_K);
  a.px_tiles = static_cast<int>((a.hw + PW_PX - 1) / PW_PX);
  a.co_tiles = static_cast<int>((d.Co + PW_CO - 1) / PW_CO);
  a.has_bias = d.has_bias ? 1 : 0;
  const int64_t blocks = static_cast<int64_t>(a.px_tiles) * a.co_tiles * g.To * d.N;
  if (blocks == 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  if (d.dtype == C3C_DTYPE_F16)
    hipLaunchKernelGGL(pointwise_conv<true>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(pointwise_conv<false>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace c3c
