// Convolutions with a 1x1 spatial kernel (stride 1 and no padding in H and
// W, one group) as per-frame matrix products on matrix cores: output frame t
// is, for each batch element,
//   y[co][p] = b[co] + sum_{k active} sum_ci w[co][ci][k] z[ci][f_k][p],
//   f_k = t * s_t + k * d_t - p_l,
// over the frames f_k of [cache; x] that exist (Eq. 2 with the source time of
// Eq. 1 and the stride of Eq. 3; a tap whose frame lies outside Z contributes
// nothing, Eq. 4).  bf16 / fp16 storage, fp32 accumulation, the bias once.
// Two users:
//   * the fast route, for temporal convolutions with a 1x1 spatial kernel
//     (Kt >= 2, any temporal stride and dilation; bf16), reading the packed
//     weights: fragment (tap k, chunk c, output fragment) is one 1 KiB block;
//   * the fallback route, for 1x1x1 calls (bf16 / fp16), reading w[co][ci].
//
// Workgroup = 160 output channels x 256 consecutive pixels of one (n, t)
// frame; eight waves of 80 channels x 64 pixels (each output row segment a
// workgroup writes is 512 contiguous bytes).  One stage = one active tap and
// one 32-channel chunk.  Its activation tile [32 ch][256 px] is copied into
// LDS as it lies in memory (pixels contiguous, as NCTHW stores them), and the
// transposing LDS read ds_read_b64_tr_b16 turns it into the matrix-core
// operand (8 consecutive channels of one pixel per lane).  The stage's
// weights are staged beside it.  Stages stream through a ring of PD register
// sets: the global loads of stage s + PD are issued while stage s computes.
// The stage count is padded to a multiple of PD with stages that read zeros,
// so every step of the loop is unconditional (the wait counts for the ring's
// loads then stay exact instead of falling back to the worst case).  Pixels
// past the end of a frame plane are loaded (from the next plane, or as zeros
// past the tensor) but only feed outputs that are never stored: a 1x1 kernel
// maps each output pixel to the same input pixel.
#include "c3c_internal.h"
#include "fuse_dev.h"

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
constexpr int PW_NT = 512;     // threads per workgroup: 2 x 4 waves
constexpr int PW_WCO = 5;      // 16-channel output fragments per wave
constexpr int PW_CO = 2 * 16 * PW_WCO;  // output channels per workgroup
static_assert(PW_CO == kPointwiseTileCo, "the tile width the dispatcher compares");
// pixels per workgroup: 4 waves along the pixels, NPF 16-pixel fragments
// each (NPF = 4: 256 pixels; NPF = 8: 512)
constexpr int pw_px(int npf) { return 4 * 16 * npf; }
// LDS bytes per staged activation channel row: pixels * 2 B + 32 B, and 128 B
// more after every 8 rows.  A transposing read serves 32 lanes at a time from
// 64 four-byte banks; those lanes read 32 B from each of rows {0..3, 8..11}
// (+4, +16 or +20 for the other halves), which the row stride (8 banks mod
// 64) and the 8-row skew (32 banks) put at banks 0, 8, 16, 24 and 32, 40,
// 48, 56: eight disjoint 8-bank groups.
constexpr int pw_pitch(int npf) { return pw_px(npf) * 2 + 32; }
constexpr int pw_row(int npf, int r) { return r * pw_pitch(npf) + (r >> 3) * 128; }
// LDS bytes per staged weight row (32 channels of one output channel): 64 B
// + 16 B, so that 8 consecutive rows read with 16-byte loads hit distinct
// 4-bank groups.
constexpr int PW_WPITCH = 80;
constexpr int pw_woff(int npf) { return pw_row(npf, PW_K); }  // weights after the activations
constexpr int pw_buf(int npf) { return pw_woff(npf) + PW_CO * PW_WPITCH; }
constexpr int PW_WPIECES = PW_CO * PW_K * 2 / 16;    // 16-byte pieces of a weight chunk
constexpr int PW_WPT = (PW_WPIECES + PW_NT - 1) / PW_NT;  // per thread
static_assert(PW_CO * PW_K * 2 <= PW_CO * PW_WPITCH, "packed weights fit the weight area");

struct PwArgs {
  const uint16_t* x;
  const uint16_t* cache;
  const uint16_t* w;      // w[co][ci] (unpacked, Kt = 1) or the packed weights
  const uint16_t* bias;
  uint16_t* y;
  int64_t hw;
  int N, Ci, Co, T, Tc, To, Z, st, dt, p_l, Kt;
  int chunks, px_tiles, co_tiles, cofrags;
  uint32_t w_bytes;
  int has_bias;
  // the fused form (FU instances; NULL when absent)
  const float* scale;
  const float* shift;
  const uint16_t* residual;
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

// PACKED: weights in matrix-core fragment order (fast route, bf16); else
// w[co][ci] (fallback, Kt = 1).  ALIGNED: every channel plane starts on a
// 16-byte boundary (H * W a multiple of 8, aligned pointers); else the
// activations are read 2 bytes at a time and the outputs stored one by one.
// FU (bf16): the fused form.  1: the residual, in the epilogue.  2: also
// the prologue on stages whose frame comes from the new chunk (applied to
// the staged registers before they go to LDS; a 1x1 kernel has no spatial
// padding, and pixels past the plane only feed outputs that are never
// stored).
template <bool F16, int PD, bool PACKED, bool ALIGNED, int PW_NPF, int FU = 0>
__global__ __launch_bounds__(PW_NT, 1) void pointwise_conv(PwArgs a) {
  constexpr int PW_PX = pw_px(PW_NPF), PW_PITCH = pw_pitch(PW_NPF);
  constexpr bool PRO = FU == 2, RES = FU >= 1;
  constexpr int PW_WOFF = pw_woff(PW_NPF), PW_BUF = pw_buf(PW_NPF);
  constexpr int SEG = PW_PX / 128;  // 16-byte row segments per thread per stage
  __shared__ __align__(16) unsigned char lds[2 * PW_BUF];
  constexpr uint32_t OOB = 0x80000000u;  // beyond every resource's size
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wco = wave & 1, wpx = wave >> 1;

  // workgroups numbered so that each of the 8 XCDs (which take workgroups
  // round-robin) runs a contiguous range of pixel tiles: neighbouring tiles
  // of a channel row are then read close together in time
  int b;
  {
    const int nb = static_cast<int>(gridDim.x), per = nb / 8, rem = nb % 8;
    const int xcd = blockIdx.x % 8, slot = blockIdx.x / 8;
    b = (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + slot;
  }
  const int pt = b % a.px_tiles;
  b /= a.px_tiles;
  const int ctile = b % a.co_tiles;
  b /= a.co_tiles;
  const int t = b % a.To;
  const int n = b / a.To;
  const int px0 = pt * PW_PX;
  // active taps (Eq. 4): source frame t s_t + k d_t - p_l inside Z; the
  // frame grows with k, so they form one range [k_lo, k_lo + ntap)
  int k_lo = 0;
  while (k_lo < a.Kt && t * a.st + k_lo * a.dt - a.p_l < 0) ++k_lo;
  int k_hi = a.Kt - 1;
  while (k_hi >= 0 && t * a.st + k_hi * a.dt - a.p_l >= a.Z) --k_hi;
  const int ntap = k_hi >= k_lo ? k_hi - k_lo + 1 : 0;
  const int nst = ntap * a.chunks;  // stages: tap outer, chunk inner

  // the channel-plane strides of the cache and of the new chunk
  const int64_t cs_c = static_cast<int64_t>(a.Tc) * a.hw, cs_x = static_cast<int64_t>(a.T) * a.hw;
  // Stages are loaded in order: tap lk, chunk lc.  The source pointer
  // (channel 32 lc of the tap's frame, pixel px0) steps by one chunk per
  // stage and only a new tap recomputes it; the stage's resource ends after
  // the chunk's last real channel's row (32-bit: a 32-channel slab fits), so
  // channels past Ci load as 0; a stage past the last has an empty resource.
  // lwrow: the stage's packed weight row, k chunks + c fragments rows in
  // (the stages' rows are consecutive).
  int lk = k_lo, lc = 0;
  const uint16_t* lp = a.x;
  uint32_t lcs = 0;     // bytes between the source's channel planes
  int64_t lstep = 0;    // elements between consecutive chunks
  bool lfx = false;     // the tap's frame comes from the new chunk
  const uint32_t lwstep = static_cast<uint32_t>(a.cofrags) * 1024u;
  uint32_t lwrow = static_cast<uint32_t>(k_lo * a.chunks) * lwstep;
  auto l_tap = [&]() __attribute__((always_inline)) {
    if (lk > k_hi) return;
    const int f = t * a.st + lk * a.dt - a.p_l;
    const bool in_cache = f < a.Tc;
    const int64_t cstride = in_cache ? cs_c : cs_x;
    lp = (in_cache ? a.cache + static_cast<int64_t>(f) * a.hw : a.x + static_cast<int64_t>(f - a.Tc) * a.hw) +
         static_cast<int64_t>(n) * a.Ci * cstride + px0;
    lcs = static_cast<uint32_t>(cstride * 2);
    lstep = PW_K * cstride;
    lfx = !in_cache;
  };
  l_tap();

  // staging: thread -> activation channel row tid / 16, pixels
  // 128 h + 8 (tid % 16) .. + 7 for h < SEG (16 lanes read 256 contiguous bytes)
  const int sch = tid >> 4, spx = (tid & 15) * 8;
  const int slds = pw_row(PW_NPF, sch) + spx * 2;
  // Weights.  Unpacked: pieces tid + 512 i -> row piece / 4, channels
  // 8 (piece % 4) .. + 7; rows past Co and channels past Ci are out-of-range
  // offsets (zeros).  Packed: piece q = 16-byte lane slot q % 64 of output
  // fragment q / 64 of the stage's (tap, chunk), fragments past the last
  // clamped to it (they feed accumulators that are never stored); stored in
  // LDS as whole fragments, 1 KiB each.
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.w), 0, static_cast<int>(a.w_bytes), 0x00020000);
  int wrow[PW_WPT], wq[PW_WPT];
  uint32_t wp_off[PW_WPT];
  bool wp_ok[PW_WPT];
#pragma unroll
  for (int i = 0; i < PW_WPT; ++i) {
    const int piece = tid + PW_NT * i;
    wrow[i] = piece >> 2;
    wq[i] = (piece & 3) * 8;
    const int frag = min(ctile * (PW_CO / 16) + piece / 64, a.cofrags - 1);
    wp_ok[i] = piece < (PW_CO / 16) * 64;
    wp_off[i] = static_cast<uint32_t>(frag) * 1024u + static_cast<uint32_t>(piece % 64) * 16u;
  }
  struct Chunk {
    u32x4 x[SEG];
    u32x4 w[PW_WPT];
    float psc, psh;  // PRO: this thread's channel's scale and shift
    bool pro;        // PRO: the stage's frame comes from the new chunk
  };
  // PRO: scale / shift of batch element n, channels past Ci read as 0
  const __amdgpu_buffer_rsrc_t ssr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(PRO && a.scale ? a.scale + static_cast<int64_t>(n) * a.Ci : a.scale), 0,
      PRO && a.scale ? a.Ci * 4 : 0, 0x00020000);
  const __amdgpu_buffer_rsrc_t shr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(PRO && a.shift ? a.shift + static_cast<int64_t>(n) * a.Ci : a.shift), 0,
      PRO && a.shift ? a.Ci * 4 : 0, 0x00020000);
  auto load_chunk = [&](Chunk& ck) __attribute__((always_inline)) {
    const bool real = lk <= k_hi;
    const uint32_t bytes = real ? static_cast<uint32_t>(min(PW_K, a.Ci - lc * PW_K) - 1) * lcs +
                                      static_cast<uint32_t>(a.hw - px0) * 2u
                                : 0u;
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(lp), 0, static_cast<int>(bytes), 0x00020000);
    if constexpr (PRO) {
      // the prologue applies to the new chunk's frames only
      const bool from_x = real && lfx;
      const uint32_t co = static_cast<uint32_t>(lc * PW_K + sch) * 4u;
      ck.pro = from_x && a.scale != nullptr;
      ck.psc = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(ssr, from_x ? co : OOB, 0, 0));
      ck.psh = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(shr, from_x ? co : OOB, 0, 0));
    }
    const uint32_t soff = static_cast<uint32_t>(sch) * lcs + static_cast<uint32_t>(spx) * 2u;
    if constexpr (ALIGNED) {
#pragma unroll
      for (int h = 0; h < SEG; ++h)
        ck.x[h] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, soff + 256u * h, 0, 0));
    } else {
#pragma unroll
      for (int h = 0; h < SEG; ++h) {
        uint32_t wd[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t o = soff + 256u * h + 4u * e;
          const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(rs, o, 0, 0);
          const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(rs, o + 2u, 0, 0);
          wd[e] = (lo & 0xffffu) | (hi << 16);
        }
        ck.x[h] = u32x4{wd[0], wd[1], wd[2], wd[3]};
      }
    }
    if constexpr (PACKED) {
      // stage (tap k, chunk c): fragment row (k * chunks + c) of the packing
#pragma unroll
      for (int i = 0; i < PW_WPT; ++i)
        ck.w[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                wrs, wp_ok[i] && real ? lwrow + wp_off[i] : OOB, 0, 0));
    } else {
      // (Kt = 1: the stage is the chunk)
#pragma unroll
      for (int i = 0; i < PW_WPT; ++i) {
        const int co = ctile * PW_CO + wrow[i], ci = lc * PW_K + wq[i];
        const bool ok = real & (wrow[i] < PW_CO) & (co < a.Co) & (ci < a.Ci);
        ck.w[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                wrs, ok ? static_cast<uint32_t>(co * a.Ci + ci) * 2u : OOB, 0, 0));
      }
    }
    lwrow += lwstep;
    if (++lc == a.chunks) {
      lc = 0;
      ++lk;
      l_tap();
    } else {
      lp += lstep;
    }
  };
  auto store_chunk = [&](const Chunk& ck, int buf) {
    unsigned char* base = lds + buf * PW_BUF;
#pragma unroll
    for (int h = 0; h < SEG; ++h) {
      // PRO: the prologue on a new-chunk stage (a workgroup-uniform test)
      u32x4 v = ck.x[h];
      if (PRO && ck.pro) v = fuse_seg8(v, ck.psc, ck.psh, true);
      *reinterpret_cast<u32x4*>(base + slds + 256 * h) = v;
    }
#pragma unroll
    for (int i = 0; i < PW_WPT; ++i) {
      if constexpr (PACKED) {
        const int piece = tid + PW_NT * i;
        if (wp_ok[i]) *reinterpret_cast<u32x4*>(base + PW_WOFF + piece * 16) = ck.w[i];
      } else {
        if (wrow[i] < PW_CO)
          *reinterpret_cast<u32x4*>(base + PW_WOFF + wrow[i] * PW_WPITCH + wq[i] * 2) = ck.w[i];
      }
    }
  };

  // transposing operand read: within each 16-lane block (channel group
  // g = l / 16), lane j names channel 8g + 4h + j / 4 at pixel group
  // 4 (j % 4) of the fragment; lane j receives channels 8g + 4h .. + 3 of
  // the fragment's pixel j
  const int j = lane & 15, g = lane >> 4;
  const int ra = pw_row(PW_NPF, 8 * g + (j >> 2)) + (wpx * 16 * PW_NPF + 4 * (j & 3)) * 2;
  auto read_a = [&](int buf, int pf) {
    const unsigned char* p = lds + buf * PW_BUF + ra + pf * 32;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 4 * PW_PITCH));
    return i16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  };
  // weight operand: lane l holds w[co = frag * 16 + l % 16][ci = 8 (l / 16) .. + 7]
  // (unpacked rows of PW_WPITCH bytes, or the packed fragment's lane slot)
  const int cof0 = ctile * PW_CO + wco * 16 * PW_WCO + (lane & 15);
  // the bias of this lane's output channel in each fragment, loaded here:
  // loaded in the epilogue, each fragment's load waited for every store
  // before it (a channel past Co, or no bias: an out-of-range offset, 0)
  float bias_v[PW_WCO];
  {
    const __amdgpu_buffer_rsrc_t brs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(a.bias), 0, a.has_bias ? a.Co * 2 : 0, 0x00020000);
#pragma unroll
    for (int cf = 0; cf < PW_WCO; ++cf)
      bias_v[cf] = from_b16(__builtin_amdgcn_raw_buffer_load_b16(brs, 2u * static_cast<uint32_t>(cof0 + 16 * cf), 0, 0),
                            F16);
  }
  const int rb = PACKED ? PW_WOFF + wco * PW_WCO * 1024 + lane * 16
                        : PW_WOFF + (wco * 16 * PW_WCO + j) * PW_WPITCH + 16 * g;
  auto read_b = [&](int buf, int cf) {
    return *reinterpret_cast<const u32x4*>(lds + buf * PW_BUF + rb +
                                           cf * (PACKED ? 1024 : 16 * PW_WPITCH));
  };

  f32x4 acc[PW_WCO][PW_NPF];
#pragma unroll
  for (int cf = 0; cf < PW_WCO; ++cf)
#pragma unroll
    for (int pf = 0; pf < PW_NPF; ++pf) acc[cf][pf] = f32x4{0.f, 0.f, 0.f, 0.f};

  Chunk ring[PD];
#pragma unroll
  for (int u = 0; u < PD; ++u) load_chunk(ring[u]);
  const int padded = (nst + PD - 1) / PD * PD;
  for (int c0 = 0; c0 < padded; c0 += PD) {
#pragma unroll
    for (int u = 0; u < PD; ++u) {
      const int c = c0 + u, buf = c & 1;
      // buffer `buf` was last read while computing chunk c - 2, which every
      // wave finished before the barrier of chunk c - 1
      store_chunk(ring[u], buf);
      load_chunk(ring[u]);  // chunk c + PD
      __syncthreads();
      i16x8 av[PW_NPF];
      u32x4 bv[PW_WCO];
#pragma unroll
      for (int pf = 0; pf < PW_NPF; ++pf) av[pf] = read_a(buf, pf);
#pragma unroll
      for (int cf = 0; cf < PW_WCO; ++cf) bv[cf] = read_b(buf, cf);
#pragma unroll
      for (int pf = 0; pf < PW_NPF; ++pf)
#pragma unroll
        for (int cf = 0; cf < PW_WCO; ++cf) acc[cf][pf] = mma<F16>(av[pf], bv[cf], acc[cf][pf]);
    }
  }

  // epilogue: lane l holds pixels 4 (l / 16) .. + 3 of output channel l % 16
  // of each fragment; bias once, one rounding, NCTHW store
  uint16_t* ybase = a.y + (static_cast<int64_t>(n) * a.Co * a.To + t) * a.hw;
#pragma unroll
  for (int cf = 0; cf < PW_WCO; ++cf) {
    const int co = cof0 + 16 * cf;
    if (co >= a.Co) continue;
    const float bb = bias_v[cf];
    uint16_t* yrow = ybase + static_cast<int64_t>(co) * a.To * a.hw;
    // RES: this fragment row's residual values, loaded as one batch before
    // its stores (branch-free: a pixel past the plane reads the row's first
    // element and is not used)
    uint2 rv[RES ? PW_NPF : 1];
    if constexpr (RES) {
      const uint16_t* rrow = a.residual ? a.residual + (yrow - a.y) : yrow;
#pragma unroll
      for (int pf = 0; pf < PW_NPF; ++pf) {
        const int p = px0 + wpx * 16 * PW_NPF + pf * 16 + 4 * g;
        if (ALIGNED) {
          rv[pf] = *reinterpret_cast<const uint2*>(rrow + (p + 4 <= a.hw ? p : 0));
        } else {
          uint16_t e[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) e[r] = rrow[p + r < a.hw ? p + r : 0];
          rv[pf] = make_uint2(e[0] | (static_cast<uint32_t>(e[1]) << 16), e[2] | (static_cast<uint32_t>(e[3]) << 16));
        }
      }
    }
#pragma unroll
    for (int pf = 0; pf < PW_NPF; ++pf) {
      const int p = px0 + wpx * 16 * PW_NPF + pf * 16 + 4 * g;
      float rr[4] = {0.f, 0.f, 0.f, 0.f};
      if (RES && a.residual) {
        // fused residual, added before the one rounding
        const uint2 r2 = rv[RES ? pf : 0];
        rr[0] = fuse_widen(r2.x & 0xffffu);
        rr[1] = fuse_widen(r2.x >> 16);
        rr[2] = fuse_widen(r2.y & 0xffffu);
        rr[3] = fuse_widen(r2.y >> 16);
      }
      uint16_t v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r)
        v[r] = F16 ? to_f16(acc[cf][pf][r] + bb + rr[r]) : to_bf16(acc[cf][pf][r] + bb + rr[r]);
      if (ALIGNED && p + 4 <= a.hw) {
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

// 1x1x1 calls (the fallback route's pointwise form, unfused) whose whole
// weight matrix fits in LDS: Co <= 160 (one output-channel tile) and at most
// kResidentChunks 32-channel chunks.  The workgroups are persistent (at most
// one per compute unit) and walk the (frame, 256-pixel tile) pairs with a
// grid stride.  Each loads the weights once, as 1 KiB matrix-core fragments
// (fragment (chunk c, output fragment f) in slot 10 c + f; lane l holds
// w[16 f + l % 16][32 c + 8 (l / 16) .. + 7], zeros past Co / Ci), so the
// stage loop fetches activations only, from HBM, through a ring of PD
// register sets that runs on across tile boundaries: the loads of the next
// tile's first chunks are in flight while a tile finishes and its outputs
// are stored.  The activation stage, its transposing LDS read and the
// epilogue are those of pointwise_conv, and so is the fused form (FU, bf16):
// the residual added before the one rounding (1), and also (2) the prologue
// applied to a new-chunk frame's staged registers before they go to LDS,
// with the tile's batch element's per-channel scale and shift (0 past Ci, so
// channels past Ci stay 0).
constexpr int kResidentChunks = 11;
constexpr int PW_RES_W = 10 * 1024 * kResidentChunks;  // resident weight bytes (max)

template <bool F16, int PD, int FU = 0>
__global__ __launch_bounds__(PW_NT, 1) void pointwise_resident(PwArgs a, int tiles_total) {
  static_assert(PD % 2 == 0, "the two LDS buffers alternate within one pass over the ring");
  static_assert(FU == 0 || !F16, "the fused form is bf16");
  constexpr bool PRO = FU == 2, RES = FU >= 1;
  constexpr int NPF = 4, PX = pw_px(NPF), PITCH = pw_pitch(NPF), SEG = PX / 128;
  constexpr int ABUF = pw_row(NPF, PW_K);  // one activation stage
  __shared__ __align__(16) unsigned char lds[PW_RES_W + 2 * ABUF];
  constexpr uint32_t OOB = 0x80000000u;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wco = wave & 1, wpx = wave >> 1;
  const int chunks = a.chunks;

  // ---- the weights, once
  {
    const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(a.w), 0, static_cast<int>(a.w_bytes), 0x00020000);
    for (int q = tid; q < chunks * 10 * 64; q += PW_NT) {
      const int l = q & 63, frag = q >> 6, c = frag / 10, f = frag % 10;
      const int co = 16 * f + (l & 15), ci = 32 * c + 8 * (l >> 4);
      const bool ok = co < a.Co && ci < a.Ci;  // Ci % 8 == 0: a slot is all in or all out
      *reinterpret_cast<u32x4*>(lds + q * 16) = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                     wrs, ok ? static_cast<uint32_t>(co * a.Ci + ci) * 2u : OOB, 0, 0));
    }
  }

  // ---- this workgroup's tiles: t = blockIdx.x + k gridDim.x; tile t is
  // (batch element, output frame, 256-pixel tile) with the pixel tile fastest
  const int ntile = (tiles_total - static_cast<int>(blockIdx.x) + static_cast<int>(gridDim.x) - 1) /
                    static_cast<int>(gridDim.x);
  const int nst = ntile * chunks;  // stages: tile outer, chunk inner
  const int64_t cs_x = static_cast<int64_t>(a.T) * a.hw, cs_c = static_cast<int64_t>(a.Tc) * a.hw;
  // Stages are loaded in order: stage g = lt chunks + lc is chunk lc of this
  // workgroup's tile lt (tile blockIdx.x + lt gridDim.x).  The source pointer
  // (channel 32 lc of the tile's frame, pixel px0) steps by one chunk per
  // stage; a new tile recomputes it (the divisions happen once per tile).
  // Its resource ends after the chunk's last real channel's row (32-bit: a
  // 32-channel slab fits).  Past the last stage, and for an output frame
  // whose one tap reads no frame of Z (Eq. 4: a left pad past the cache, or
  // a right pad), the resource is empty (zeros: the output is the bias alone).
  int lt = 0, lc = 0;
  const uint16_t* lp = a.x;
  uint32_t lcs = 0, lpx = 0;  // bytes between channel planes; pixel bytes left in the plane
  int64_t lstep = 0;          // elements between consecutive chunks
  bool lact = false;
  bool lpro = false;  // PRO: the tile's frame comes from the new chunk
  int lsc = 0;        // PRO: the tile's batch element's first scale / shift index
  auto l_tile = [&]() __attribute__((always_inline)) {
    const int t = static_cast<int>(blockIdx.x) + lt * static_cast<int>(gridDim.x);
    const int pt = t % a.px_tiles, nt = t / a.px_tiles;
    const int o = nt % a.To, n = nt / a.To;
    const int f = o * a.st - a.p_l;  // Kt = 1: the one tap's source frame
    lact = lt < ntile && f >= 0 && f < a.Z;
    const bool in_cache = lact && f < a.Tc;
    lpro = PRO && lact && !in_cache && a.scale != nullptr;
    lsc = n * a.Ci;
    const int64_t cstride = in_cache ? cs_c : cs_x;
    const int64_t px0 = static_cast<int64_t>(pt) * PX;
    lp = lact ? (in_cache ? a.cache + static_cast<int64_t>(f) * a.hw : a.x + static_cast<int64_t>(f - a.Tc) * a.hw) +
                    static_cast<int64_t>(n) * a.Ci * cstride + px0
              : a.x;
    lcs = static_cast<uint32_t>(cstride * 2);
    lpx = lact ? static_cast<uint32_t>(a.hw - px0) * 2u : 0u;
    lstep = PW_K * cstride;
  };
  l_tile();
  const int sch = tid >> 4, spx = (tid & 15) * 8;
  const int slds = pw_row(NPF, sch) + spx * 2;
  // PRO: scale / shift [N][Ci] as fp32 resources; this thread's channel of
  // the stage (32 lc + sch) reads 0 past Ci
  const uint32_t sbytes = PRO && a.scale ? static_cast<uint32_t>(a.N * a.Ci) * 4u : 0u;
  const __amdgpu_buffer_rsrc_t ssr = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.scale), 0,
                                                                       static_cast<int>(sbytes), 0x00020000);
  const __amdgpu_buffer_rsrc_t shr = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.shift), 0,
                                                                       static_cast<int>(sbytes), 0x00020000);
  struct Slot {
    u32x4 x[SEG];
    float psc, psh;
    bool pro;
  };
  auto load = [&](Slot& sl) __attribute__((always_inline)) {
    u32x4(&x)[SEG] = sl.x;
    if constexpr (PRO) {
      const int c = lc * PW_K + sch;
      const uint32_t off = lpro && c < a.Ci ? static_cast<uint32_t>(lsc + c) * 4u : OOB;
      sl.pro = lpro;
      sl.psc = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(ssr, off, 0, 0));
      sl.psh = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(shr, off, 0, 0));
    }
    const uint32_t bytes = lact ? static_cast<uint32_t>(min(PW_K, a.Ci - lc * PW_K) - 1) * lcs + lpx : 0u;
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(lp), 0, static_cast<int>(bytes), 0x00020000);
    const uint32_t soff = static_cast<uint32_t>(sch) * lcs + static_cast<uint32_t>(spx) * 2u;
#pragma unroll
    for (int h = 0; h < SEG; ++h)
      x[h] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, soff + 256u * h, 0, 0));
    if (++lc == chunks) {
      lc = 0;
      ++lt;
      l_tile();
    } else {
      lp += lstep;
    }
  };
  auto store = [&](const Slot& sl, int buf) {
#pragma unroll
    for (int h = 0; h < SEG; ++h) {
      u32x4 v = sl.x[h];
      if (PRO && sl.pro) v = fuse_seg8(v, sl.psc, sl.psh, true);  // workgroup-uniform
      *reinterpret_cast<u32x4*>(lds + PW_RES_W + buf * ABUF + slds + 256 * h) = v;
    }
  };
  const int j = lane & 15, gq = lane >> 4;
  const int ra = pw_row(NPF, 8 * gq + (j >> 2)) + (wpx * 16 * NPF + 4 * (j & 3)) * 2;
  // the bias of this lane's output channel in each fragment, the same for
  // every tile: loaded once here (loaded in each tile's epilogue, every
  // fragment's load waited for the tile's earlier stores; a channel past Co,
  // or no bias: an out-of-range offset, 0)
  float bias_v[PW_WCO];
  {
    const __amdgpu_buffer_rsrc_t brs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(a.bias), 0, a.has_bias ? a.Co * 2 : 0, 0x00020000);
#pragma unroll
    for (int cf = 0; cf < PW_WCO; ++cf)
      bias_v[cf] = from_b16(
          __builtin_amdgcn_raw_buffer_load_b16(brs, 2u * static_cast<uint32_t>(wco * 16 * PW_WCO + 16 * cf + j), 0, 0),
          F16);
  }
  auto read_a = [&](int buf, int pf) {
    const unsigned char* p = lds + PW_RES_W + buf * ABUF + ra + pf * 32;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 4 * PITCH));
    return i16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  };
  auto read_b = [&](int c, int cf) {
    return *reinterpret_cast<const u32x4*>(lds + ((c * 10 + wco * PW_WCO + cf) * 64 + lane) * 16);
  };

  f32x4 acc[PW_WCO][NPF];
#pragma unroll
  for (int cf = 0; cf < PW_WCO; ++cf)
#pragma unroll
    for (int pf = 0; pf < NPF; ++pf) acc[cf][pf] = f32x4{0.f, 0.f, 0.f, 0.f};

  Slot ring[PD];
#pragma unroll
  for (int u = 0; u < PD; ++u) load(ring[u]);
  const int padded = (nst + PD - 1) / PD * PD;
  int ct = 0, c = 0;  // tile ordinal and chunk of the stage being computed
  for (int g0 = 0; g0 < padded; g0 += PD) {
#pragma unroll
    for (int u = 0; u < PD; ++u) {
      const int buf = u & 1;  // (g0 + u) & 1: PD is even
      // buffer `buf` was last read while computing stage g - 2, which every
      // wave finished before the barrier of stage g - 1
      store(ring[u], buf);
      load(ring[u]);  // stage g + PD
      __syncthreads();
      // the tile's last chunk (workgroup-uniform): its outputs are stored
      // after the products; RES: the tile's residual values are loaded
      // first, so that they arrive during the products
      const bool last = c == chunks - 1 && ct < ntile;
      int64_t toff = 0;  // element offset of output channel 0 of the tile's (n, o) plane, pixel 0
      int64_t tp0 = 0;   // the tile's first pixel
      if (last) {
        const int t = static_cast<int>(blockIdx.x) + ct * static_cast<int>(gridDim.x);
        const int pt = t % a.px_tiles, nt = t / a.px_tiles;
        const int o = nt % a.To, n = nt / a.To;
        toff = (static_cast<int64_t>(n) * a.Co * a.To + o) * a.hw;
        tp0 = static_cast<int64_t>(pt) * PX + wpx * 16 * NPF + 4 * gq;
      }
      uint2 rv[RES ? PW_WCO : 1][RES ? NPF : 1];
      if (RES && last && a.residual) {
#pragma unroll
        for (int cf = 0; cf < PW_WCO; ++cf) {
          const int co = wco * 16 * PW_WCO + 16 * cf + j;
          const int64_t roff = toff + static_cast<int64_t>(co < a.Co ? co : 0) * a.To * a.hw;
#pragma unroll
          for (int pf = 0; pf < NPF; ++pf) {
            const int64_t p = tp0 + pf * 16;  // hw % 8 == 0: four pixels all in or all out
            rv[cf][pf] = *reinterpret_cast<const uint2*>(a.residual + roff + (p < a.hw ? p : 0));
          }
        }
      }
      i16x8 av[NPF];
      u32x4 bv[PW_WCO];
#pragma unroll
      for (int pf = 0; pf < NPF; ++pf) av[pf] = read_a(buf, pf);
#pragma unroll
      for (int cf = 0; cf < PW_WCO; ++cf) bv[cf] = read_b(c, cf);
#pragma unroll
      for (int pf = 0; pf < NPF; ++pf)
#pragma unroll
        for (int cf = 0; cf < PW_WCO; ++cf) acc[cf][pf] = mma<F16>(av[pf], bv[cf], acc[cf][pf]);
      // bias once, one rounding (the residual added before it), NCTHW store;
      // the accumulators start again from zero
      if (last) {
#pragma unroll
        for (int cf = 0; cf < PW_WCO; ++cf) {
          const int co = wco * 16 * PW_WCO + 16 * cf + j;
          const float bb = bias_v[cf];
          uint16_t* yrow = a.y + toff + static_cast<int64_t>(co) * a.To * a.hw;
#pragma unroll
          for (int pf = 0; pf < NPF; ++pf) {
            const int64_t p = tp0 + pf * 16;
            if (co < a.Co && p < a.hw) {  // hw % 8 == 0: four pixels all in or all out
              float rr[4] = {0.f, 0.f, 0.f, 0.f};
              if (RES && a.residual) {
                const uint2 r2 = rv[RES ? cf : 0][RES ? pf : 0];
                rr[0] = fuse_widen(r2.x & 0xffffu);
                rr[1] = fuse_widen(r2.x >> 16);
                rr[2] = fuse_widen(r2.y & 0xffffu);
                rr[3] = fuse_widen(r2.y >> 16);
              }
              uint16_t v[4];
#pragma unroll
              for (int r = 0; r < 4; ++r)
                v[r] = F16 ? to_f16(acc[cf][pf][r] + bb + rr[r]) : to_bf16(acc[cf][pf][r] + bb + rr[r]);
              *reinterpret_cast<uint2*>(yrow + p) =
                  make_uint2(v[0] | (static_cast<uint32_t>(v[1]) << 16), v[2] | (static_cast<uint32_t>(v[3]) << 16));
            }
            acc[cf][pf] = f32x4{0.f, 0.f, 0.f, 0.f};
          }
        }
      }
      if (++c == chunks) {
        c = 0;
        ++ct;
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

namespace {

// one launch of pointwise_conv: the ring depth that pads the largest stage
// count of any output frame least (4, 3 or 2), the template instance by
// element type, weight layout and alignment
template <bool PACKED>
hipError_t launch_pw(const Geo& g, PwArgs a, bool f16, bool al, hipStream_t s, int fused,
                     LaunchInfo* info) {
  const c3c_conv_desc& d = g.d;
  a.co_tiles = static_cast<int>((d.Co + PW_CO - 1) / PW_CO);
  // Fast route, aligned: 512-pixel workgroups (twice the products per
  // staged weight chunk; 1.4x on a 384->768 120x208 temporal conv) unless
  // that leaves fewer workgroups than half the compute units.  Otherwise
  // 256-pixel ones: the unpacked-weight and unaligned instances would spill
  // at 512 (with 8 waves a wave has 256 registers), and on the 1x1x1
  // shortcut the wide tile measured no faster.
  const int64_t tiles512 = (a.hw + pw_px(8) - 1) / pw_px(8);
  const bool wide = PACKED && al && tiles512 * a.co_tiles * g.To * d.N * 2 >= device_compute_units();
  const int px = wide ? pw_px(8) : pw_px(4);
  a.px_tiles = static_cast<int>((a.hw + px - 1) / px);
  const int64_t blocks = static_cast<int64_t>(a.px_tiles) * a.co_tiles * g.To * d.N;
  if (info) {
    info->kernel = C3C_KERNEL_POINTWISE;
    info->tile_co = PW_CO;
    info->tile_h = 0;
    info->tile_w = px;
    info->workgroups = blocks;
    return hipSuccess;
  }
  if (blocks == 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  int ntap = 0;
  for (int64_t t = 0; t < g.To; ++t) {
    int nt = 0;
    for (int64_t k = 0; k < d.Kt; ++k) {
      const int64_t f = t * d.stride_t + k * d.dil_t - g.p_l;
      nt += f >= 0 && f < g.Z;
    }
    ntap = nt > ntap ? nt : ntap;
  }
  const int nst = ntap * a.chunks;
  // ring depth: 2 for 512-pixel workgroups (their staging registers leave
  // no room for more); for 256-pixel ones, the one of 4, 3, 2 that pads the
  // stage count least
  int pd = 2;
  if (!wide) {
    pd = 4;
    for (int cand : {3, 2})
      if ((nst + cand - 1) / cand * cand < (nst + pd - 1) / pd * pd) pd = cand;
  }
  const dim3 grid(static_cast<unsigned>(blocks)), block(PW_NT);
#define C3C_PW(F, P, A, NPF, FU)                                                               \
  if (f16 == F && pd == P && al == A && (NPF == 8) == wide && fused == FU) {                    \
    hipLaunchKernelGGL((pointwise_conv<F, P, PACKED, A, NPF, FU>), grid, block, 0, s, a);      \
    return hipGetLastError();                                                                  \
  }
  if constexpr (PACKED) {  // fast route: bf16, any alignment
    C3C_PW(false, 2, true, 4, 0) C3C_PW(false, 3, true, 4, 0) C3C_PW(false, 4, true, 4, 0)
    C3C_PW(false, 2, false, 4, 0) C3C_PW(false, 3, false, 4, 0) C3C_PW(false, 4, false, 4, 0)
    C3C_PW(false, 2, true, 8, 0)
    C3C_PW(false, 2, true, 4, 1) C3C_PW(false, 3, true, 4, 1) C3C_PW(false, 4, true, 4, 1)
    C3C_PW(false, 2, false, 4, 1) C3C_PW(false, 3, false, 4, 1) C3C_PW(false, 4, false, 4, 1)
    C3C_PW(false, 2, true, 8, 1)
    C3C_PW(false, 2, true, 4, 2) C3C_PW(false, 3, true, 4, 2) C3C_PW(false, 4, true, 4, 2)
    C3C_PW(false, 2, false, 4, 2) C3C_PW(false, 3, false, 4, 2) C3C_PW(false, 4, false, 4, 2)
    C3C_PW(false, 2, true, 8, 2)
  } else {  // fallback: bf16 / fp16, aligned (pointwise_eligible)
    C3C_PW(false, 2, true, 4, 0) C3C_PW(false, 3, true, 4, 0) C3C_PW(false, 4, true, 4, 0)
    C3C_PW(true, 2, true, 4, 0) C3C_PW(true, 3, true, 4, 0) C3C_PW(true, 4, true, 4, 0)
    C3C_PW(false, 2, true, 4, 1) C3C_PW(false, 3, true, 4, 1) C3C_PW(false, 4, true, 4, 1)
    C3C_PW(false, 2, true, 4, 2) C3C_PW(false, 3, true, 4, 2) C3C_PW(false, 4, true, 4, 2)
  }
#undef C3C_PW
  return hipErrorInvalidValue;
}

PwArgs common_args(const Geo& g, const void* x, const void* cache, const void* bias, void* y) {
  const c3c_conv_desc& d = g.d;
  PwArgs a;
  a.x = static_cast<const uint16_t*>(x);
  a.cache = static_cast<const uint16_t*>(cache);
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
  a.dt = static_cast<int>(d.dil_t);
  a.p_l = static_cast<int>(g.p_l);
  a.Kt = static_cast<int>(d.Kt);
  a.chunks = static_cast<int>((d.Ci + PW_K - 1) / PW_K);
  a.has_bias = d.has_bias ? 1 : 0;
  a.scale = a.shift = nullptr;
  a.residual = nullptr;
  return a;
}

}  // namespace

hipError_t launch_pointwise(const Geo& g, const void* x, const void* cache, const void* w,
                            const void* bias, void* y, hipStream_t s, const Fuse& fu,
                            LaunchInfo* info) {
  PwArgs a = common_args(g, x, cache, bias, y);
  const bool f16 = g.d.dtype == C3C_DTYPE_F16;
  // calls whose weights fit in LDS (the fused form: bf16): the persistent
  // resident-weight kernel
  if ((!fu.any() || !f16) && g.d.Co <= PW_CO && a.chunks <= kResidentChunks && g.d.N * g.To > 0) {
    a.w = static_cast<const uint16_t*>(w);
    a.w_bytes = static_cast<uint32_t>(g.d.Co * g.d.Ci * 2);
    a.cofrags = 0;
    a.co_tiles = 1;
    a.px_tiles = static_cast<int>((a.hw + pw_px(4) - 1) / pw_px(4));
    const int64_t tiles = static_cast<int64_t>(a.px_tiles) * g.To * g.d.N;
    const int64_t cus = device_compute_units();
    const int64_t blocks = tiles < cus ? tiles : cus;
    if (info) {
      info->kernel = C3C_KERNEL_POINTWISE;
      info->tile_co = PW_CO;
      info->tile_h = 0;
      info->tile_w = pw_px(4);
      info->workgroups = blocks;
      return hipSuccess;
    }
    if (tiles > 0x7fffffff) return hipErrorInvalidConfiguration;
    a.scale = fu.scale;
    a.shift = fu.shift;
    a.residual = fu.residual;  // launch_fallback checked its 8-byte alignment
    const dim3 grid(static_cast<unsigned>(blocks)), block(PW_NT);
    if (f16)
      hipLaunchKernelGGL((pointwise_resident<true, 4>), grid, block, 0, s, a, static_cast<int>(tiles));
    else if (fu.pro())
      hipLaunchKernelGGL((pointwise_resident<false, 4, 2>), grid, block, 0, s, a, static_cast<int>(tiles));
    else if (fu.residual)
      hipLaunchKernelGGL((pointwise_resident<false, 4, 1>), grid, block, 0, s, a, static_cast<int>(tiles));
    else
      hipLaunchKernelGGL((pointwise_resident<false, 4>), grid, block, 0, s, a, static_cast<int>(tiles));
    return hipGetLastError();
  }
  a.w = static_cast<const uint16_t*>(w);
  a.w_bytes = static_cast<uint32_t>(g.d.Co * g.d.Ci * 2);
  a.cofrags = 0;
  a.scale = fu.scale;
  a.shift = fu.shift;
  a.residual = fu.residual;
  // launch_fallback checked the residual's 8-byte alignment
  return launch_pw<false>(g, a, g.d.dtype == C3C_DTYPE_F16, true, s, fu.pro() ? 2 : fu.residual ? 1 : 0,
                          info);
}

hipError_t launch_fast_tap1x1(const Geo& g, const void* x, const void* cache, const void* wpack,
                              const void* bias, void* y, hipStream_t s, const Fuse& fu,
                              LaunchInfo* info) {
  const c3c_conv_desc& d = g.d;
  const PackDims p = pack_dims(d);
  // 32-bit buffer offsets: one 32-channel chunk of a source frame and the
  // packed weights must each span less than 2 GiB
  const int64_t frames = d.T > d.Tc ? d.T : d.Tc;
  if (static_cast<int64_t>(PW_K) * frames * d.H * d.W * 2 >= 0x7fffffff || p.elems() * 2 >= 0x7fffffff)
    return hipErrorInvalidValue;
  PwArgs a = common_args(g, x, cache, bias, y);
  a.w = static_cast<const uint16_t*>(wpack);
  a.w_bytes = static_cast<uint32_t>(p.elems() * 2);
  a.cofrags = static_cast<int>(p.cofrags);
  a.scale = fu.scale;
  a.shift = fu.shift;
  a.residual = fu.residual;
  const bool al = (d.H * d.W) % 8 == 0 && aligned(x, 16) && (cache == nullptr || aligned(cache, 16)) &&
                  aligned(y, 8) && (fu.residual == nullptr || aligned(fu.residual, 8));
  return launch_pw<true>(g, a, false, al, s, fu.pro() ? 2 : fu.residual ? 1 : 0, info);
}

}  // namespace c3c
