// Fast route, shared parts: the packed-weight layout and its repack / unpack
// kernels, the dispatch of one fast call, and the fp32 kernel.  The bf16
// kernel lives in conv_bf16.hip.
//
// The fp32 kernel is the same cache-aware lowering of a causal Conv3D (paper
// Sec. 4, Eq. 2 and Eq. 4, Alg. 1) as one implicit-GEMM kernel on gfx950 fp32
// matrix cores, in a simpler form (single-buffered LDS, no prefetch): fp32
// calls are small validation workloads.
//
// The paper evaluates each active temporal tap k as a batched Conv2D over the
// frames [z_l, z_h) of Z = [C; X]_T, folded into the batch, and sums the taps
// into an accumulator before adding the bias once.  Here the fold is only an
// index map: a workgroup owns an output tile (one frame o, a BH x BW block of
// pixels, a block of output channels) and, for every tap whose Eq. 4 interval
// contains o, reads source frame o + delta_k straight from the cache or from
// the new chunk (no concatenated copy of Z), so all taps accumulate in fp32
// registers.  The bias is added once in the epilogue.
//
// GEMM view per output frame: D[co][px] = sum_K A[co][K] * B[K][px] with
// K = (tap kt, kh, kw, input channel).  A (weights) comes pre-packed in
// matrix-core fragment order; B (activations) is staged through LDS as a halo
// tile [BH+KS-1][BW+KS-1][channels], channel-innermost, so that each lane
// reads its K-contiguous operand with one LDS load and the KS x KS spatial
// offsets (a 3x3 kernel with pad 1, or 1x1) are address shifts into the same
// tile.  Source frame of tap k for output frame o: o s_t + k d_t - p_l (the
// temporal stride is 1 for 3x3 kernels).
#include "c3c_internal.h"

namespace c3c {

PackDims pack_dims(const c3c_conv_desc& d) {
  PackDims p;
  const bool f32 = d.dtype == C3C_DTYPE_F32;
  p.rows = f32 ? 32 : 16;
  p.kpl = f32 ? 1 : 8;
  p.kstep = (64 / p.rows) * p.kpl;
  p.taps = d.Kt * d.Kh * d.Kw;
  p.chunks = (d.Ci + p.kstep - 1) / p.kstep;
  p.cofrags = (d.Co + p.rows - 1) / p.rows;
  return p;
}

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- repack
// packed index (tap, chunk, cofrag, lane, e) <-> w[co][ci][tap]
template <typename T>
__global__ __launch_bounds__(256) void repack_kernel(const T* __restrict__ w, T* __restrict__ wp,
                                                     int64_t total, int64_t Ci, int64_t Co,
                                                     int64_t taps, int64_t chunks,
                                                     int64_t cofrags, int rows, int kpl) {
  const int kstep = (64 / rows) * kpl;
  for (int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; idx < total;
       idx += static_cast<int64_t>(gridDim.x) * 256) {
    int64_t r = idx;
    const int e = static_cast<int>(r % kpl);
    r /= kpl;
    const int lane = static_cast<int>(r % 64);
    r /= 64;
    const int64_t cf = r % cofrags;
    r /= cofrags;
    const int64_t ch = r % chunks;
    const int64_t tap = r / chunks;
    const int64_t co = cf * rows + lane % rows;
    const int64_t ci = ch * kstep + (lane / rows) * kpl + e;
    T v = T(0);
    if (co < Co && ci < Ci) v = w[(co * Ci + ci) * taps + tap];
    wp[idx] = v;
  }
}

// 16-bit weights, fragment geometry rows = 16, kpl = 8 (32 input channels
// per chunk): one workgroup per (chunk, output fragment) block.  The block's
// 16 output channels x 32 input channels x all taps are contiguous runs of
// w (32 * taps elements per output channel), read coalesced into LDS; each
// thread then writes whole 16-byte lane slots (8 consecutive input channels
// of one output channel at one tap) of the block's fragments, one 1 KiB
// fragment per 64 threads.  Channels past Ci / Co are zeros.  vec: w is
// 16-byte aligned and Ci * taps a multiple of 8, so a full chunk's runs are
// read as 16-byte pieces (the tail chunk, and other calls, element by
// element).
constexpr int kRepackMaxTaps = 48;
__global__ __launch_bounds__(256) void repack_block16(const uint16_t* __restrict__ w,
                                                      u32x4* __restrict__ wp, int64_t Ci,
                                                      int64_t Co, int taps, int64_t chunks,
                                                      int64_t cofrags, int vec) {
  __shared__ __align__(16) uint16_t tile[16 * 32 * kRepackMaxTaps];
  const int64_t cf = blockIdx.x % cofrags, ch = blockIdx.x / cofrags;
  const int row = 32 * taps;  // elements of one output channel's run
  const int64_t ci0 = ch * 32;
  const int64_t ci_n = Ci - ci0 < 32 ? Ci - ci0 : 32;  // real input channels of the chunk
  if (vec && ci_n == 32) {
    const int nv = row / 8;  // 16-byte pieces of a run
    for (int q = threadIdx.x; q < 16 * nv; q += 256) {
      const int r = q / nv, u = q - r * nv;
      const int64_t co = cf * 16 + r;
      *reinterpret_cast<u32x4*>(tile + r * row + 8 * u) =
          co < Co ? *reinterpret_cast<const u32x4*>(w + (co * Ci + ci0) * taps + 8 * u) : u32x4{0u, 0u, 0u, 0u};
    }
  } else {
    for (int q = threadIdx.x; q < 16 * row; q += 256) {
      const int r = q / row, u = q - r * row;
      const int64_t co = cf * 16 + r;
      const bool ok = co < Co && u < ci_n * taps;
      tile[q] = ok ? w[(co * Ci + ci0) * taps + u] : static_cast<uint16_t>(0);
    }
  }
  __syncthreads();
  // thread -> (tap t, lane L): lane L holds output channel L % 16, input
  // channels 8 (L / 16) .. + 7
  for (int q = threadIdx.x; q < taps * 64; q += 256) {
    const int t = q >> 6, L = q & 63;
    const int base = ((L & 15) * 32 + 8 * (L >> 4)) * taps + t;
    uint32_t v[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      v[e] = static_cast<uint32_t>(tile[base + (2 * e) * taps]) |
             (static_cast<uint32_t>(tile[base + (2 * e + 1) * taps]) << 16);
    wp[((t * chunks + ch) * cofrags + cf) * 64 + L] = u32x4{v[0], v[1], v[2], v[3]};
  }
}

template <typename T>
__global__ __launch_bounds__(256) void unpack_kernel(const T* __restrict__ wp, T* __restrict__ w,
                                                     int64_t total, int64_t Ci, int64_t taps,
                                                     int64_t chunks, int64_t cofrags, int rows,
                                                     int kpl) {
  const int64_t kstep = (64 / rows) * kpl;
  for (int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; idx < total;
       idx += static_cast<int64_t>(gridDim.x) * 256) {
    const int64_t tap = idx % taps;
    const int64_t ci = (idx / taps) % Ci;
    const int64_t co = idx / (taps * Ci);
    const int64_t ch = ci / kstep, rem = ci % kstep;
    const int64_t lane = co % rows + rows * (rem / kpl);
    const int64_t e = rem % kpl;
    const int64_t cf = co / rows;
    w[idx] = wp[((((tap * chunks + ch) * cofrags + cf) * 64 + lane) * kpl) + e];
  }
}

// ---------------------------------------------------------------- conversions
__device__ inline uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// ---------------------------------------------------------------- matrix-core policy
// fp32: v_mfma_f32_32x32x2_f32, each lane supplies 1 K value.
// Output fragment: lane l holds D[row][col = l % 32] for the 16 rows
// row = 8 * (r / 4) + 4 * (l / 32) + (r % 4), r = 0..15.
template <typename T>
struct Mma;

template <>
struct Mma<float> {
  static constexpr int KPL = 1, KSTEP = 2, BKC = 16, PIXS = 17;
  typedef float frag;
  static __device__ inline frag zero() { return 0.f; }
  static __device__ inline frag load(const float* p) { return *p; }
  static __device__ inline f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  static __device__ inline float to_f(float v) { return v; }
  static __device__ inline float from_f(float v) { return v; }
};

struct FastArgs {
  const void* x;
  const void* cache;
  const void* wpack;
  const void* bias;
  void* y;
  int64_t Ci, Co, T, Tc, H, W;
  int64_t Kt, dt, st, p_l, Z, To;
  int64_t chunks, cofrags;
  int tiles_co, tiles_w, tiles_h;
  int has_bias;
};

// Workgroup tile: BCO = 32 * CO_FRAGS * WAVES_CO output channels by
// BH rows x (32 * BWF) columns of one output frame.  Wave (wco, wpx) owns
// CO_FRAGS x PX_FRAGS 32x32 accumulator fragments.
template <typename T, int CO_FRAGS, int PX_FRAGS, int WAVES_CO, int WAVES_PX, int BH, int BWF, int KS>
__global__ __launch_bounds__(64 * WAVES_CO * WAVES_PX) void fast_conv3d(FastArgs a) {
  using M = Mma<T>;
  static_assert(WAVES_PX * PX_FRAGS == BH * BWF, "pixel fragments must tile the block");
  constexpr int NT = 64 * WAVES_CO * WAVES_PX;
  constexpr int BW = 32 * BWF;
  constexpr int TW = BW + KS - 1, TH = BH + KS - 1;  // halo tile, pad (KS - 1) / 2
  constexpr int PAD = (KS - 1) / 2;
  constexpr int BKC = M::BKC, PIXS = M::PIXS, KSTEP = M::KSTEP, KPL = M::KPL;
  __shared__ __align__(16) T tile[TH * TW * PIXS];

  const T* __restrict__ x = static_cast<const T*>(a.x);
  const T* __restrict__ cache = static_cast<const T*>(a.cache);
  const typename M::frag* __restrict__ wp = static_cast<const typename M::frag*>(a.wpack);
  const T* __restrict__ bias = static_cast<const T*>(a.bias);
  T* __restrict__ y = static_cast<T*>(a.y);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wco = wave % WAVES_CO, wpx = wave / WAVES_CO;

  int64_t id = blockIdx.x;
  const int ct = static_cast<int>(id % a.tiles_co);
  id /= a.tiles_co;
  const int tw = static_cast<int>(id % a.tiles_w);
  id /= a.tiles_w;
  const int th = static_cast<int>(id % a.tiles_h);
  id /= a.tiles_h;
  const int64_t o = id % a.To, n = id / a.To;
  const int h0 = th * BH, w0 = tw * BW;
  const int64_t hw = a.H * a.W;
  const int cofrag0 = (ct * WAVES_CO + wco) * CO_FRAGS;

  f32x16 acc[CO_FRAGS][PX_FRAGS];
#pragma unroll
  for (int i = 0; i < CO_FRAGS; ++i)
#pragma unroll
    for (int j = 0; j < PX_FRAGS; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  for (int64_t k = 0; k < a.Kt; ++k) {
    // Eq. 4: tap k is active for this frame iff its source frame lies in Z.
    const int64_t f = o * a.st + k * a.dt - a.p_l;
    if (f < 0 || f >= a.Z) continue;
    const T* src;
    int64_t cstride;
    if (f < a.Tc) {
      src = cache + (n * a.Ci * a.Tc + f) * hw;
      cstride = a.Tc * hw;
    } else {
      src = x + (n * a.Ci * a.T + (f - a.Tc)) * hw;
      cstride = a.T * hw;
    }
    for (int64_t c0 = 0; c0 < a.Ci; c0 += BKC) {
      __syncthreads();
      // stage the halo tile: rows h0-1 .. h0+BH, cols w0-1 .. w0+BW, BKC channels
      for (int e = tid; e < BKC * TH * TW; e += NT) {
        const int cc = e % TW, rr = (e / TW) % TH, ch = e / (TW * TH);
        const int gh = h0 - PAD + rr, gw = w0 - PAD + cc;
        T v = T(0);
        if (c0 + ch < a.Ci && gh >= 0 && gh < a.H && gw >= 0 && gw < a.W)
          v = src[(c0 + ch) * cstride + static_cast<int64_t>(gh) * a.W + gw];
        tile[(rr * TW + cc) * PIXS + ch] = v;
      }
      __syncthreads();
      // A spatial tap's weight fragments (its BKC / KSTEP K-steps) are loaded
      // one tap ahead of its products, into a second register set, so that
      // no product waits for a weight load issued just before it.
      constexpr int NKS = BKC / KSTEP;
      typename M::frag wa[NKS][CO_FRAGS], wb[NKS][CO_FRAGS];
      auto load_wt = [&](int ij, typename M::frag (&w)[NKS][CO_FRAGS]) {
        const int64_t tap = k * KS * KS + ij;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          const int64_t chunk = c0 / KSTEP + ks;
#pragma unroll
          for (int cf = 0; cf < CO_FRAGS; ++cf) {
            const int cofrag = cofrag0 + cf;
            w[ks][cf] = chunk < a.chunks && cofrag < a.cofrags
                            ? wp[((tap * a.chunks + chunk) * a.cofrags + cofrag) * 64 + lane]
                            : M::zero();
          }
        }
      };
      auto products = [&](int ij, const typename M::frag (&w)[NKS][CO_FRAGS]) {
        const int ki = ij / KS, kj = ij % KS;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          const int64_t chunk = c0 / KSTEP + ks;
          if (chunk >= a.chunks) break;
          typename M::frag bf[PX_FRAGS];
#pragma unroll
          for (int pf = 0; pf < PX_FRAGS; ++pf) {
            const int q = wpx * PX_FRAGS + pf;
            const int r = q / BWF, cb = (q % BWF) * 32;
            bf[pf] = M::load(&tile[((r + ki) * TW + cb + (lane & 31) + kj) * PIXS + ks * KSTEP +
                                   (lane >> 5) * KPL]);
          }
#pragma unroll
          for (int cf = 0; cf < CO_FRAGS; ++cf)
#pragma unroll
            for (int pf = 0; pf < PX_FRAGS; ++pf) acc[cf][pf] = M::mma(w[ks][cf], bf[pf], acc[cf][pf]);
        }
      };
      load_wt(0, wa);
#pragma unroll 1
      for (int ij = 0; ij < KS * KS; ij += 2) {
        if (ij + 1 < KS * KS) load_wt(ij + 1, wb);
        products(ij, wa);
        if (ij + 1 < KS * KS) {
          if (ij + 2 < KS * KS) load_wt(ij + 2, wa);
          products(ij + 1, wb);
        }
      }
    }
  }

  // epilogue: bias once, round to the storage type, NCTHW store
  const int64_t Ho = a.H, Wo = a.W;
#pragma unroll
  for (int cf = 0; cf < CO_FRAGS; ++cf) {
    const int cofrag = cofrag0 + cf;
#pragma unroll
    for (int pf = 0; pf < PX_FRAGS; ++pf) {
      const int q = wpx * PX_FRAGS + pf;
      const int h = h0 + q / BWF, wc = w0 + (q % BWF) * 32 + (lane & 31);
      if (h >= Ho || wc >= Wo) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t co = static_cast<int64_t>(cofrag) * 32 + 8 * (r / 4) + 4 * (lane >> 5) + (r & 3);
        if (co >= a.Co) continue;
        float v = acc[cf][pf][r];
        if (a.has_bias) v += M::to_f(bias[co]);
        y[((n * a.Co + co) * a.To + o) * Ho * Wo + static_cast<int64_t>(h) * Wo + wc] = M::from_f(v);
      }
    }
  }
}

template <typename T, int CO_FRAGS, int PX_FRAGS, int WAVES_CO, int WAVES_PX, int BH, int BWF, int KS>
hipError_t run_fast(const Geo& g, FastArgs a, hipStream_t s, LaunchInfo* info) {
  constexpr int BCO = 32 * CO_FRAGS * WAVES_CO, BW = 32 * BWF;
  a.tiles_co = static_cast<int>((g.d.Co + BCO - 1) / BCO);
  a.tiles_w = static_cast<int>((g.Wo + BW - 1) / BW);
  a.tiles_h = static_cast<int>((g.Ho + BH - 1) / BH);
  const int64_t blocks = static_cast<int64_t>(a.tiles_co) * a.tiles_w * a.tiles_h * g.To * g.d.N;
  if (info) {
    info->kernel = C3C_KERNEL_FAST_F32;
    info->tile_co = BCO;
    info->tile_h = BH;
    info->tile_w = BW;
    info->workgroups = blocks;
    return hipSuccess;
  }
  if (blocks == 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((fast_conv3d<T, CO_FRAGS, PX_FRAGS, WAVES_CO, WAVES_PX, BH, BWF, KS>),
                     dim3(static_cast<unsigned>(blocks)), dim3(64 * WAVES_CO * WAVES_PX), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_repack(const Geo& g, const void* w, void* wpack, hipStream_t s) {
  const PackDims p = pack_dims(g.d);
  const int64_t total = p.elems();
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (g.d.dtype == C3C_DTYPE_F32)
    hipLaunchKernelGGL(repack_kernel<float>, dim3(blocks), dim3(256), 0, s,
                       static_cast<const float*>(w), static_cast<float*>(wpack), total, g.d.Ci,
                       g.d.Co, p.taps, p.chunks, p.cofrags, p.rows, p.kpl);
  else if (p.rows == 16 && p.kpl == 8 && p.taps <= kRepackMaxTaps &&
           p.chunks * p.cofrags <= 0x7fffffff && (reinterpret_cast<uintptr_t>(wpack) & 15u) == 0)
    hipLaunchKernelGGL(repack_block16, dim3(static_cast<unsigned>(p.chunks * p.cofrags)), dim3(256),
                       0, s, static_cast<const uint16_t*>(w), static_cast<u32x4*>(wpack), g.d.Ci,
                       g.d.Co, static_cast<int>(p.taps), p.chunks, p.cofrags,
                       ((reinterpret_cast<uintptr_t>(w) & 15u) == 0 && (g.d.Ci * p.taps) % 8 == 0) ? 1 : 0);
  else
    hipLaunchKernelGGL(repack_kernel<uint16_t>, dim3(blocks), dim3(256), 0, s,
                       static_cast<const uint16_t*>(w), static_cast<uint16_t*>(wpack), total,
                       g.d.Ci, g.d.Co, p.taps, p.chunks, p.cofrags, p.rows, p.kpl);
  return hipGetLastError();
}

hipError_t launch_unpack(const Geo& g, const void* wpack, void* w, hipStream_t s) {
  const PackDims p = pack_dims(g.d);
  const int64_t total = g.d.Co * g.d.Ci * p.taps;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (g.d.dtype == C3C_DTYPE_F32)
    hipLaunchKernelGGL(unpack_kernel<float>, dim3(blocks), dim3(256), 0, s,
                       static_cast<const float*>(wpack), static_cast<float*>(w), total, g.d.Ci,
                       p.taps, p.chunks, p.cofrags, p.rows, p.kpl);
  else
    hipLaunchKernelGGL(unpack_kernel<uint16_t>, dim3(blocks), dim3(256), 0, s,
                       static_cast<const uint16_t*>(wpack), static_cast<uint16_t*>(w), total,
                       g.d.Ci, p.taps, p.chunks, p.cofrags, p.rows, p.kpl);
  return hipGetLastError();
}

hipError_t launch_fast(const Geo& g, const void* x, const void* cache, const void* wpack,
                       const void* bias, void* y, void* cache_out, void* ws, int64_t ws_bytes,
                       hipStream_t s, const Fuse& fu, LaunchInfo* info) {
  const PackDims p = pack_dims(g.d);
  FastArgs a;
  a.x = x; a.cache = cache; a.wpack = wpack; a.bias = bias; a.y = y;
  a.Ci = g.d.Ci; a.Co = g.d.Co; a.T = g.d.T; a.Tc = g.d.Tc; a.H = g.d.H; a.W = g.d.W;
  a.Kt = g.d.Kt; a.dt = g.d.dil_t; a.st = g.d.stride_t; a.p_l = g.p_l; a.Z = g.Z; a.To = g.To;
  a.chunks = p.chunks; a.cofrags = p.cofrags;
  a.has_bias = g.d.has_bias ? 1 : 0;
  a.tiles_co = a.tiles_w = a.tiles_h = 0;
  // the fast route's two spatial forms: 3x3 / stride 1 / pad 1, and 1x1
  const bool one = g.d.Kh == 1;
  hipError_t e;
  if (g.d.dtype == C3C_DTYPE_BF16) {
    if (one) {
      // Two kernels: the 4-wave 192 x 128 kernel (aligned calls; 1.2-1.5x
      // the pointwise kernel at Co = 768 and 384) unless its padded output
      // channels exceed the 160-channel pointwise tile's by more than 10%
      // (Co = 96, 160, 256, 320 stay on the pointwise kernel) or its tiles
      // leave half the compute units idle.  The fused form (prologue /
      // residual) is in the pointwise kernel only.
      const int64_t pad_tap = (g.d.Co + kTap1x1TileCo - 1) / kTap1x1TileCo * kTap1x1TileCo;
      const int64_t pad_pw = (g.d.Co + kPointwiseTileCo - 1) / kPointwiseTileCo * kPointwiseTileCo;
      if (!fu.any() && 10 * pad_tap <= 11 * pad_pw && tap1x1_eligible(g, x, cache, y) &&
          2 * tap1x1_blocks(g) >= device_compute_units()) {
        bool written = false;
        e = launch_tap1x1(g, x, cache, wpack, bias, y, cache_out, &written, s, info);
        if (e != hipSuccess || written || info) return e;
      } else
        e = launch_fast_tap1x1(g, x, cache, wpack, bias, y, s, fu, info);
    } else if (!fu.any() && head_eligible(g, x, cache, y)) {
      // few output channels (a decoder's RGB head): the spatial taps as N
      bool written = false;
      e = launch_head(g, x, cache, wpack, bias, y, cache_out, &written, s, info);
      if (e != hipSuccess || written || info) return e;
    } else {
      bool written = false;
      e = launch_fast_bf16(g, x, cache, wpack, bias, y, cache_out, ws, ws_bytes, &written, s, fu,
                           info);
      if (e != hipSuccess || written || info) return e;
    }
  } else if (g.Wo <= 32) {
    // narrow frames: 4 x 32-pixel tiles (a 64-pixel-wide tile would compute
    // half its columns past the frame)
    e = one ? run_fast<float, 1, 1, 1, 4, 4, 1, 1>(g, a, s, info)
            : run_fast<float, 1, 1, 1, 4, 4, 1, 3>(g, a, s, info);
  } else {
    e = one ? run_fast<float, 1, 2, 1, 4, 4, 2, 1>(g, a, s, info)
            : run_fast<float, 1, 2, 1, 4, 4, 2, 3>(g, a, s, info);
  }
  if (e != hipSuccess || info) return e;
  return launch_cache_copy(g, x, cache, cache_out, s, fu);
}

}  // namespace c3c
