// Fast route, bf16, 1x1 spatial kernel: temporal convolutions (kernel Kt x 1
// x 1, any temporal stride and dilation) as per-frame matrix products on
// gfx950 matrix cores, several workgroups per compute unit.
//
// Output frame t of batch element n is
//   y[co][p] = b[co] + sum_{k active} sum_ci w[co][ci][k] z[ci][f_k][p],
//   f_k = t * s_t + k * d_t - p_l,
// over the frames f_k of [cache; x] that exist (Eq. 2 with the source time of
// Eq. 1 and the stride of Eq. 3; Eq. 4 drops the others), bias once.
//
// Workgroup = 192 output channels x 128 consecutive pixels of one (n, t)
// frame, 4 waves side by side along the output channels, each 48 channels x
// all 128 pixels: 3 x 8 accumulator fragments of v_mfma_f32_16x16x32_bf16
// (activations as the A operand, lane l holding 4 consecutive pixels of
// channel l % 16).  Every wave needs different weights, so no weight byte is
// fetched twice per workgroup; the activation tile is shared through LDS.
// A stage is short (24 products per wave), so the tile is sized for several
// workgroups per compute unit (19 KB of LDS, 162 registers a lane: three)
// whose stages cover each other's memory waits: 1.2-1.5x faster than 320-
// pixel tiles at one workgroup per unit, which read less L2 per product.
// A stage is one active tap and one 32-channel chunk:
//   * its activation tile [32 ch][128 px] is copied into LDS as it lies in
//     memory (pixels contiguous) and read back with the transposing
//     ds_read_b64_tr_b16, which gives each lane 8 consecutive channels of one
//     pixel;
//   * its weights are the packed fragments (tap, chunk, output fragment), one
//     16-byte load per lane each, straight from L2 into registers.
// Pipeline: during stage s the waves issue the weights of stage s + 1 and the
// activation loads of stage s + 2, compute stage s, then write stage s + 1's
// activations (loaded during stage s - 1) into the other LDS buffer, and one
// barrier publishes it.  The stage loop is unrolled by two (register sets
// alternate), the stage count padded to even with stages that read zeros.
// Pixels past the end of a frame plane are loaded (the next plane, or zeros
// past the tensor) but only feed outputs that are never stored.
// The new cache (the last L frames of [cache; x]) is written from the staging
// registers: by the output-channel tile 0 workgroup of the first output frame
// that reads each of its frames, as that frame's tiles go to LDS, when every
// new-cache frame is read by some output frame (the launcher checks;
// otherwise the caller copies it).
// Calls with one output frame take the chunk-stage form further down.
//
// Requires H * W a multiple of 8 and 16-byte-aligned x / cache, 8-byte y.
#include "c3c_internal.h"

#include <type_traits>

namespace c3c {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int TK = 32;                 // input channels per stage (one matrix-core K step)
constexpr int TPX = 128;               // pixels per workgroup
constexpr int WCO = 3, NPF = TPX / 16; // fragments per wave: 48 channels x 128 pixels
constexpr int TCO = 4 * WCO * 16;      // output channels per workgroup
static_assert(TCO == kTap1x1TileCo, "the tile width the dispatcher compares");
// LDS offset of staged channel row r: pitch 256 B + 32 B (8 banks mod 64),
// and 128 B more after every 8 rows.  A transposing read serves 32 lanes at
// a time from 64 four-byte banks; those lanes read 32 B from each of rows
// {0..3, 8..11} (+4, +16 or +20 for the other halves), which start at banks
// 0, 8, 16, 24 and 32, 40, 48, 56: eight disjoint 8-bank groups.
constexpr int TPITCH = TPX * 2 + 32;
constexpr int row_off(int r) { return r * TPITCH + (r >> 3) * 128; }
constexpr int TBUF = row_off(TK);
constexpr int TSEG = TK * TPX / 8;     // 16-byte segments of a stage tile
constexpr int TSPT = TSEG / 256;       // per thread
static_assert(TSEG % 256 == 0, "the stage tile splits evenly over the threads");

struct TapArgs {
  const uint16_t* x;
  const uint16_t* cache;
  const u32x4* wpack;
  const uint16_t* bias;
  uint16_t* y;
  int64_t hw;
  int N, Ci, Co, T, Tc, To, Z, st, dt, p_l, Kt;
  int chunks, cofrags, px_tiles, co_tiles, nblocks;
  uint32_t wpack_bytes;
  int has_bias;
  // the new cache, written by the kernel when write_cache (L frames)
  uint16_t* cache_out;
  int L, write_cache;
};

__global__ __launch_bounds__(256, 2) void conv_tap1x1(TapArgs a) {
  __shared__ __align__(16) unsigned char lds[2 * TBUF];
  constexpr uint32_t OOB = 0x80000000u;  // beyond every resource's size
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wco = wave;  // output-channel slice of this wave

  // workgroups numbered so that each of the 8 XCDs (which take workgroups
  // round-robin) runs a contiguous range: the output-channel tiles of a pixel
  // tile (which read the same activations) run close together
  int b;
  {
    const int per = a.nblocks / 8, rem = a.nblocks % 8;
    const int xcd = static_cast<int>(blockIdx.x) % 8, slot = static_cast<int>(blockIdx.x) / 8;
    b = (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + slot;
  }
  const int ctile = b % a.co_tiles;
  b /= a.co_tiles;
  const int pt = b % a.px_tiles;
  b /= a.px_tiles;
  const int t = b % a.To;
  const int n = b / a.To;
  const int px0 = pt * TPX;

  // active taps (Eq. 4): one contiguous range [k_lo, k_lo + ntap)
  int k_lo = 0;
  while (k_lo < a.Kt && t * a.st + k_lo * a.dt - a.p_l < 0) ++k_lo;
  int k_hi = a.Kt - 1;
  while (k_hi >= 0 && t * a.st + k_hi * a.dt - a.p_l >= a.Z) --k_hi;
  const int ntap = k_hi >= k_lo ? k_hi - k_lo + 1 : 0;
  const int nst = ntap * a.chunks;  // tap outer, chunk inner
  // taps whose frame this workgroup writes to the new cache: output-channel
  // tile 0, a frame of the new cache, and read by no earlier output frame
  // (t' < t with t' s_t = f + p_l - k d_t); the launcher allows this only
  // for Kt <= 32
  uint32_t cwk = 0;
  if (a.write_cache && ctile == 0)
    for (int k = k_lo; k <= k_hi; ++k) {
      const int f = t * a.st + k * a.dt - a.p_l;
      if (f < a.Z - a.L) continue;
      bool before = false;
      for (int k2 = 0; k2 < a.Kt; ++k2) {
        const int kd = f + a.p_l - k2 * a.dt;
        if (kd >= 0 && kd % a.st == 0 && kd / a.st < t) before = true;
      }
      if (!before) cwk |= 1u << k;
    }
  const int padded = (nst + 1) & ~1;

  // activation stages are loaded in order: (ak, ac) is the tap and channel
  // chunk of the next one, ap its channel 32 ac of frame f_ak at pixel px0.
  // The pointer steps by one chunk per stage and only a new tap recomputes
  // it (a stage's scalar work is a few additions).  Its source is a buffer
  // resource that ends after the chunk's last real channel's row (32-bit:
  // a 32-channel slab fits), empty past the last stage.
  const int64_t cs_c = static_cast<int64_t>(a.Tc) * a.hw, cs_x = static_cast<int64_t>(a.T) * a.hw;
  int ak = k_lo, ac = 0;
  const uint16_t* ap = a.x;
  uint32_t acs = 0;   // bytes between the source's channel planes
  int64_t astep = 0;  // elements between consecutive chunks
  auto act_tap = [&]() __attribute__((always_inline)) {
    if (ak > k_hi) return;
    const int f = t * a.st + ak * a.dt - a.p_l;
    const bool in_cache = f < a.Tc;
    const int64_t cstride = in_cache ? cs_c : cs_x;
    ap = (in_cache ? a.cache + static_cast<int64_t>(f) * a.hw : a.x + static_cast<int64_t>(f - a.Tc) * a.hw) +
         static_cast<int64_t>(n) * a.Ci * cstride + px0;
    acs = static_cast<uint32_t>(cstride * 2);
    astep = TK * cstride;
  };
  act_tap();
  auto next_rsrc = [&](uint32_t& cs) __attribute__((always_inline)) {
    const bool real = ak <= k_hi;
    const uint32_t bytes = real ? static_cast<uint32_t>(min(TK, a.Ci - ac * TK) - 1) * acs +
                                      static_cast<uint32_t>(a.hw - px0) * 2u
                                : 0u;
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(ap), 0, static_cast<int>(bytes), 0x00020000);
    cs = acs;
    if (++ac == a.chunks) {
      ac = 0;
      ++ak;
      act_tap();
    } else {
      ap += astep;
    }
    return rs;
  };

  // staging: segment q = tid + 256 i of the tile -> channel row q / 16,
  // pixels 8 (q % 16) .. + 7 (consecutive lanes read consecutive 16 bytes)
  uint32_t s_row[TSPT], s_px[TSPT], s_lds[TSPT];
#pragma unroll
  for (int i = 0; i < TSPT; ++i) {
    const int q = tid + 256 * i, r = q / (TPX / 8), c = q % (TPX / 8);
    s_row[i] = static_cast<uint32_t>(r);
    s_px[i] = static_cast<uint32_t>(c) * 16u;
    s_lds[i] = static_cast<uint32_t>(row_off(r) + c * 16);
  }
  auto load_act = [&](u32x4 (&v)[TSPT]) {
    uint32_t cs;
    const __amdgpu_buffer_rsrc_t rs = next_rsrc(cs);
#pragma unroll
    for (int i = 0; i < TSPT; ++i)
      v[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, s_row[i] * cs + s_px[i], 0, 0));
  };
  // the next stage's activations (stages are stored in order: tap sk,
  // chunk sc) into LDS buffer buf; a stage whose frame goes to the new cache
  // [N][Ci][L][H*W] (frame f is its frame f - (Z - L)) is also written there
  // from the same registers (the chunk's real rows, pixels inside the plane)
  const int64_t cl = static_cast<int64_t>(a.L) * a.hw;
  int sk = k_lo, sc = 0;
  auto store_act = [&](const u32x4 (&v)[TSPT], int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < TSPT; ++i) *reinterpret_cast<u32x4*>(lds + buf * TBUF + s_lds[i]) = v[i];
    const int k = sk, c0 = sc * TK;
    if (++sc == a.chunks) {
      sc = 0;
      ++sk;
    }
    if (cwk != 0 && k <= k_hi && ((cwk >> k) & 1u)) {
      const int f = t * a.st + k * a.dt - a.p_l;
      const uint32_t ccs = static_cast<uint32_t>(cl * 2);
      const uint32_t cbytes = static_cast<uint32_t>(min(TK, a.Ci - c0) - 1) * ccs + static_cast<uint32_t>(a.hw) * 2u;
      const __amdgpu_buffer_rsrc_t crs = __builtin_amdgcn_make_buffer_rsrc(
          a.cache_out + (static_cast<int64_t>(n) * a.Ci + c0) * cl + static_cast<int64_t>(f - (a.Z - a.L)) * a.hw,
          0, static_cast<int>(cbytes), 0x00020000);
#pragma unroll
      for (int i = 0; i < TSPT; ++i) {
        const uint32_t px = px0 + s_px[i] / 2u;
        __builtin_amdgcn_raw_buffer_store_b128(v[i], crs,
                                               px < static_cast<uint32_t>(a.hw) ? s_row[i] * ccs + px * 2u : OOB, 0, 0);
      }
    }
  };

  // weights: fragment (tap k, chunk c, output fragment ctile 12 + wco 3 + cf),
  // clamped to the last packed fragment (padding rows are never stored); an
  // out-of-range offset (zeros) past the last stage
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<u32x4*>(a.wpack), 0, static_cast<int>(a.wpack_bytes), 0x00020000);
  uint32_t w_off[WCO];
#pragma unroll
  for (int cf = 0; cf < WCO; ++cf)
    w_off[cf] = static_cast<uint32_t>(min(ctile * (TCO / 16) + wco * WCO + cf, a.cofrags - 1)) * 1024u +
                static_cast<uint32_t>(lane) * 16u;
  // the bias of this lane's output channel in each fragment, loaded here:
  // loaded in the epilogue, each fragment's load waited for every store
  // before it (a channel past Co, or no bias: an out-of-range offset, 0)
  float bias_v[WCO];
  {
    const __amdgpu_buffer_rsrc_t brs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(a.bias), 0, a.has_bias ? a.Co * 2 : 0, 0x00020000);
#pragma unroll
    for (int cf = 0; cf < WCO; ++cf) {
      const uint32_t co = static_cast<uint32_t>(ctile * TCO + wco * 16 * WCO + cf * 16 + (lane & 15));
      bias_v[cf] = __uint_as_float(static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b16(brs, 2u * co, 0, 0))
                                   << 16);
    }
  }
  // weights are loaded in order: stage ws is tap k_lo + ws / chunks, chunk
  // ws % chunks, packed row k_lo * chunks + ws (wrow its byte offset)
  int ws = 0;
  uint32_t wrow = static_cast<uint32_t>(k_lo * a.chunks * a.cofrags) * 1024u;
  const uint32_t wstep = static_cast<uint32_t>(a.cofrags) * 1024u;
  auto load_w = [&](u32x4 (&v)[WCO]) __attribute__((always_inline)) {
    const bool real = ws < nst;
#pragma unroll
    for (int cf = 0; cf < WCO; ++cf)
      v[cf] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                            wrs, real ? wrow + w_off[cf] : OOB, 0, 0));
    ++ws;
    wrow += wstep;
  };

  // transposing operand read: within each 16-lane block (channel group
  // g = l / 16), lane j names channel 8g + 4h + j / 4 at pixel group
  // 4 (j % 4) of the fragment; lane j receives channels 8g + 4h .. + 3 of
  // the fragment's pixel j (h = 0, 1: the two halves)
  const int j = lane & 15, g = lane >> 4;
  const int ra = row_off(8 * g + (j >> 2)) + 4 * (j & 3) * 2;
  auto read_a = [&](int buf, int pf) {
    const unsigned char* p = lds + buf * TBUF + ra + pf * 32;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 4 * TPITCH));
    return i16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  };

  f32x4 acc[WCO][NPF];
#pragma unroll
  for (int cf = 0; cf < WCO; ++cf)
#pragma unroll
    for (int pf = 0; pf < NPF; ++pf) acc[cf][pf] = f32x4{0.f, 0.f, 0.f, 0.f};

  // prologue: weights of stage 0, activations of stages 0 and 1 in flight,
  // stage 0 into LDS buffer 0
  u32x4 act0[TSPT], act1[TSPT];
  u32x4 w0[WCO], w1[WCO];
  load_w(w0);
  load_act(act0);
  load_act(act1);
  store_act(act0, 0);
  __syncthreads();

  // one stage: weights of s + 1 and activations of s + 2 issued (their
  // register sets were consumed in stage s - 1), the products of s, then
  // s + 1's activations into the other buffer (last read in stage s - 1,
  // before its barrier)
  auto stage = [&](int buf, const u32x4 (&w_cur)[WCO], u32x4 (&w_nxt)[WCO], u32x4 (&a_free)[TSPT],
                   const u32x4 (&a_next)[TSPT]) {
    load_w(w_nxt);
    load_act(a_free);
    i16x8 av[NPF];
#pragma unroll
    for (int pf = 0; pf < NPF; ++pf) av[pf] = read_a(buf, pf);
#pragma unroll
    for (int pf = 0; pf < NPF; ++pf)
#pragma unroll
      for (int cf = 0; cf < WCO; ++cf)
        acc[cf][pf] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            __builtin_bit_cast(bf16x8, av[pf]), __builtin_bit_cast(bf16x8, w_cur[cf]), acc[cf][pf], 0, 0, 0);
    store_act(a_next, buf ^ 1);
    __syncthreads();
  };
  for (int s = 0; s < padded; s += 2) {
    stage(0, w0, w1, act0, act1);
    stage(1, w1, w0, act1, act0);
  }

  // epilogue: lane l holds pixels 4 (l / 16) .. + 3 of output channel l % 16
  // of each fragment; bias once, one round-to-nearest-even, NCTHW store
  uint16_t* ybase = a.y + (static_cast<int64_t>(n) * a.Co * a.To + t) * a.hw;
#pragma unroll
  for (int cf = 0; cf < WCO; ++cf) {
    const int co = ctile * TCO + wco * 16 * WCO + cf * 16 + (lane & 15);
    if (co >= a.Co) continue;
    const float bb = bias_v[cf];
    uint16_t* yrow = ybase + static_cast<int64_t>(co) * a.To * a.hw;
#pragma unroll
    for (int pf = 0; pf < NPF; ++pf) {
      const int p = px0 + pf * 16 + 4 * g;
      if (p >= a.hw) continue;
      const uint32_t v01 = __builtin_bit_cast(
          uint32_t, __builtin_convertvector((f32x2{acc[cf][pf][0] + bb, acc[cf][pf][1] + bb}), bf16x2));
      const uint32_t v23 = __builtin_bit_cast(
          uint32_t, __builtin_convertvector((f32x2{acc[cf][pf][2] + bb, acc[cf][pf][3] + bb}), bf16x2));
      // H * W is a multiple of 8, so 4 pixels from a multiple of 4 stay in the plane
      *reinterpret_cast<uint2*>(yrow + p) = make_uint2(v01, v23);
    }
  }
}

// ---------------------------------------------------------------------------
// Chunk-stage form, for calls with one output frame (a decoder's first
// temporal upsampling).  The same 192 x 128 tile of one output frame, but one
// stage is one 32-channel chunk of every tap (up to 3): its source frames
// (one slot per tap, frame F0 + k d_t with F0 = t s_t - p_l) are staged into
// LDS together, the weights of all taps of the chunk loaded together, so a
// stage carries up to 3 x 24 products per wave and its barrier is paid over
// three times the work.  A slot whose frame lies outside [0, Z) (Eq. 4) or
// whose tap is >= Kt is staged as zeros with zero weights.
// Staging: the activation tiles go from memory straight into LDS (buffer
// loads with the LDS destination, 16 bytes a lane; no registers), each
// [32 ch][128 px] tile as 32 rows of 256 bytes whose 16-byte segments are
// permuted within the row (segment s of row r at s ^ sw(r)), so that the
// transposing reads stay free of bank conflicts without padding.
// Pipeline: three LDS buffers and three weight register sets; during chunk c
// the waves issue chunk c + 2's weights and tiles into set and buffer
// (c + 2) % 3 (last used in chunk c - 1), run chunk c's products from buffer
// c % 3 (its first slot read before the previous barrier), then wait for
// their own share of chunk c + 1's tiles (issued a stage earlier) and meet at
// one barrier.  The explicit wait and a plain barrier (no release fence) let
// chunk c + 2's loads stay in flight across it.
// The new cache: the output-channel tile 0 workgroup of the first output
// frame that reads a new-cache frame copies it from LDS (the launcher checks
// that every new-cache frame is read by some output frame).
constexpr int KTG = 3;       // taps this form holds weights for
constexpr int GTILE = 8192;  // bytes of one staged [32 ch][128 px] tile
// segment permutation of row r: rows {0..3, 8..11} (and {4..7, 12..15}),
// which one transposing read pass serves, land in 8 distinct 32-byte bank
// groups
__device__ __forceinline__ uint32_t seg_swizzle(uint32_t r) { return ((r & 3u) | (((r >> 3) & 1u) << 2)) << 1; }
typedef __attribute__((address_space(3))) void lds_void;

__global__ __launch_bounds__(256, 1) void conv_tap1x1_chunk(TapArgs a) {
  constexpr int NR = KTG;  // frame slots, one per tap
  // three stage buffers, each its own array: the compiler then knows that a
  // load into one does not write what is read from another (a single array
  // makes it wait for every load into LDS before any LDS read)
  __shared__ __align__(16) unsigned char lds0[NR * GTILE];
  __shared__ __align__(16) unsigned char lds1[NR * GTILE];
  __shared__ __align__(16) unsigned char lds2[NR * GTILE];
  auto bufp = [&](auto B) -> unsigned char* { return B.value == 0 ? lds0 : B.value == 1 ? lds1 : lds2; };
  constexpr uint32_t OOB = 0x80000000u;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);

  // XCD-contiguous numbering, as above: the output-channel tiles of a pixel
  // tile run close together
  int b;
  {
    const int per = a.nblocks / 8, rem = a.nblocks % 8;
    const int xcd = static_cast<int>(blockIdx.x) % 8, slot = static_cast<int>(blockIdx.x) / 8;
    b = (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + slot;
  }
  const int ctile = b % a.co_tiles;
  b /= a.co_tiles;
  const int pt = b % a.px_tiles;
  // one output frame (t = 0: the launcher takes this form only for To = 1)
  const int n = b / a.px_tiles;
  const int px0 = pt * TPX;

  // slot r (tap r) reads frame r d_t - p_l; live: r < Kt and the frame in
  // [0, Z); cwm: live and a frame of the new cache (no earlier output frame
  // has read it: there is none)
  const int F0 = -a.p_l;
  auto slot_frame = [&](int r) { return F0 + r * a.dt; };
  uint32_t live = 0, cwm = 0;
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const int f = slot_frame(r);
    if (r >= a.Kt || f < 0 || f >= a.Z) continue;
    live |= 1u << r;
    if (a.write_cache && ctile == 0 && f >= a.Z - a.L) cwm |= 1u << r;
  }

  // staging: this wave's two 1 KiB blocks of a tile are rows 4 (4 i + wv)
  // .. + 3; lane l fills row 4 (4 i + wv) + l / 16, LDS segment l % 16, with
  // the row's segment (l % 16) ^ sw(row) (pixels 8 of it .. + 7)
  uint32_t d_row[2], d_px[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const uint32_t r = static_cast<uint32_t>(4 * (4 * i + wv) + (lane >> 4));
    d_row[i] = r;
    d_px[i] = ((static_cast<uint32_t>(lane) & 15u) ^ seg_swizzle(r)) * 16u;
  }
  const int64_t cs_c = static_cast<int64_t>(a.Tc) * a.hw, cs_x = static_cast<int64_t>(a.T) * a.hw;
  // slot r's source, built once: every channel of its frame from pixel px0
  // (32-bit sizes: the launcher checks the extent), empty (zeros) for a slot
  // that is not live.  A stage adds its chunk's 32 channel planes to the
  // lanes' offsets, so the channels past Ci and a chunk past the last are
  // out-of-range offsets and read zeros.
  __amdgpu_buffer_rsrc_t srs[NR];
  uint32_t scs[NR];
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const int f = slot_frame(r);
    const bool real = (live >> r) & 1u;
    const bool in_cache = f < a.Tc;
    const int64_t cstride = in_cache ? cs_c : cs_x;
    const uint16_t* base = in_cache ? a.cache : a.x;
    const int64_t off = static_cast<int64_t>(in_cache ? f : f - a.Tc) * a.hw +
                        static_cast<int64_t>(n) * a.Ci * cstride + px0;
    scs[r] = static_cast<uint32_t>(cstride * 2);
    const uint32_t bytes =
        real ? static_cast<uint32_t>(a.Ci - 1) * scs[r] + static_cast<uint32_t>(a.hw - px0) * 2u : 0u;
    srs[r] = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(real ? base + off : a.x), 0,
                                               static_cast<int>(bytes), 0x00020000);
  }
  // chunk c's tiles into the LDS buffer at L (2 NR loads per lane)
  auto stage_act = [&](int c, unsigned char* L) {
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      const uint32_t add = static_cast<uint32_t>(c * TK) * scs[r];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(srs[r], (lds_void*)(L + r * GTILE + (4 * i + wv) * 1024), 16,
                                                 d_row[i] * scs[r] + d_px[i] + add, 0, 0, 0);
    }
  };
  // the new cache [N][Ci][L][H*W] (frame f is its frame f - (Z - L)):
  // chunk c's cache slots copied from the LDS buffer at L, 16 bytes a lane,
  // rows as staged (segment permutation undone on the way out)
  // (one resource over batch element n's new cache, every channel and frame,
  // built once: 32-bit sizes, the launcher checks the extent; a channel past
  // Ci is an out-of-range offset and its stores are dropped)
  const int64_t cl = static_cast<int64_t>(a.L) * a.hw;
  const uint32_t ccs = static_cast<uint32_t>(cl * 2);
  const __amdgpu_buffer_rsrc_t crs = __builtin_amdgcn_make_buffer_rsrc(
      cwm != 0 ? a.cache_out + static_cast<int64_t>(n) * a.Ci * cl : a.y, 0,
      cwm != 0 ? static_cast<int>(static_cast<uint32_t>(a.Ci) * ccs) : 0, 0x00020000);
  auto copy_cache = [&](int c, const unsigned char* L) {
    const uint32_t cadd = static_cast<uint32_t>(c * TK) * ccs;
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      if (!((cwm >> r) & 1u)) continue;
      const uint32_t fo = static_cast<uint32_t>(slot_frame(r) - (a.Z - a.L)) * static_cast<uint32_t>(a.hw) * 2u + cadd;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const uint32_t q = static_cast<uint32_t>(tid + 256 * i), row = q >> 4, ls = q & 15u;
        const u32x4 v = *reinterpret_cast<const u32x4*>(L + r * GTILE + q * 16);
        const uint32_t px = px0 + (ls ^ seg_swizzle(row)) * 8u;
        __builtin_amdgcn_raw_buffer_store_b128(v, crs,
                                               px < static_cast<uint32_t>(a.hw) ? row * ccs + px * 2 + fo : OOB, 0, 0);
      }
    }
  };

  // weights: fragment (tap k, chunk c, output fragment ctile 12 + wv 3 + cf),
  // clamped to the last packed fragment (padding rows are never stored); an
  // out-of-range offset (zeros) for k >= Kt or a chunk past the last
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<u32x4*>(a.wpack), 0, static_cast<int>(a.wpack_bytes), 0x00020000);
  uint32_t w_off[WCO];
#pragma unroll
  for (int cf = 0; cf < WCO; ++cf)
    w_off[cf] = static_cast<uint32_t>(min(ctile * (TCO / 16) + wv * WCO + cf, a.cofrags - 1)) * 1024u +
                static_cast<uint32_t>(lane) * 16u;
  // the bias of this lane's output channel in each fragment, loaded here (as
  // in the kernel above)
  float bias_v[WCO];
  {
    const __amdgpu_buffer_rsrc_t brs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(a.bias), 0, a.has_bias ? a.Co * 2 : 0, 0x00020000);
#pragma unroll
    for (int cf = 0; cf < WCO; ++cf) {
      const uint32_t co = static_cast<uint32_t>(ctile * TCO + wv * 16 * WCO + cf * 16 + (lane & 15));
      bias_v[cf] = __uint_as_float(static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b16(brs, 2u * co, 0, 0))
                                   << 16);
    }
  }
  auto load_w = [&](int c, u32x4 (&v)[KTG][WCO]) {
#pragma unroll
    for (int k = 0; k < KTG; ++k) {
      const bool real = k < a.Kt && c < a.chunks;
      const uint32_t row = static_cast<uint32_t>((k * a.chunks + c) * a.cofrags) * 1024u;
#pragma unroll
      for (int cf = 0; cf < WCO; ++cf)
        v[k][cf] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                 wrs, real ? row + w_off[cf] : OOB, 0, 0));
    }
  };

  // transposing operand read: within each 16-lane block g = l / 16, lane j
  // reads 8 bytes of channel row 8g + 4h + j / 4 (h = 0, 1) at pixel
  // 16 pf + 4 (j % 4) of the tile, i.e. staged segment 2 pf + (j % 4) / 2;
  // with the even permutation sw(row) that is byte
  // row 256 + 32 (pf ^ sw(row) / 2) + 8 (j % 4) = ra ^ 32 pf.
  // (z: a zero the compiler cannot see through, fresh each stage, so that
  // the addresses are formed where they are used rather than held in
  // registers across the loop for every buffer and slot)
  const int j16 = lane & 15, g = lane >> 4;
  const uint32_t rrow = static_cast<uint32_t>(8 * g + (j16 >> 2));
  const uint32_t ra = rrow * 256u + 16u * seg_swizzle(rrow) + 8u * static_cast<uint32_t>(j16 & 3);
  auto read_a = [&](const unsigned char* L, int r, i16x8 (&av)[NPF], uint32_t z) {
#pragma unroll
    for (int pf = 0; pf < NPF; ++pf) {
      const unsigned char* p = L + r * GTILE + ((ra + z) ^ (32u * pf));
      const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
      const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 4 * 256));
      av[pf] = i16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    }
  };

  f32x4 acc[WCO][NPF];
#pragma unroll
  for (int cf = 0; cf < WCO; ++cf)
#pragma unroll
    for (int pf = 0; pf < NPF; ++pf) acc[cf][pf] = f32x4{0.f, 0.f, 0.f, 0.f};

  // wait until at most n vector-memory operations of this wave are
  // outstanding (the LDS and export counters left alone)
#define C3C_VMCNT(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | (7 << 4) | (15 << 8))
  auto barrier = [] { asm volatile("s_barrier" ::: "memory"); };

  // One stage: chunk c's products from LDS buffer B with weight set B, slot
  // by slot.  A slot's operands are read during the previous slot's
  // products (one read after each of the first 2 x NPF products; slot 0's
  // before the previous barrier), slot r into operand set r % 2.  No
  // instruction moves across a slot's end.
  u32x4 w[3][KTG][WCO];
  i16x8 avs[2][NPF];
  auto stage = [&](int c, auto B) {
    constexpr int b0 = decltype(B)::value, b1 = (b0 + 1) % 3, b2 = (b0 + 2) % 3;
    unsigned char* const cur_b = bufp(B);
    unsigned char* const next_b = bufp(std::integral_constant<int, b1>{});
    unsigned char* const fill_b = bufp(std::integral_constant<int, b2>{});
    uint32_t z;
    asm volatile("v_mov_b32 %0, 0" : "=v"(z));
    if (cwm != 0 && c < a.chunks) copy_cache(c, cur_b);
    load_w(c + 2, w[b2]);
    stage_act(c + 2, fill_b);
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      const i16x8(&cur)[NPF] = avs[r & 1];
      if (r + 1 < NR) read_a(cur_b, r + 1, avs[(r + 1) & 1], z);
#pragma unroll
      for (int pf = 0; pf < NPF; ++pf)
#pragma unroll
        for (int cf = 0; cf < WCO; ++cf)
          acc[cf][pf] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(bf16x8, cur[pf]), __builtin_bit_cast(bf16x8, w[b0][r][cf]), acc[cf][pf], 0, 0, 0);
      if (r + 1 < NR) {
#pragma unroll
        for (int q = 0; q < 2 * NPF; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // a matrix-core product
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // an LDS read
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    read_a(next_b, 0, avs[0], z);
    // this wave's loads of chunk c + 1 (issued a stage ago, the tiles after
    // the weights) have landed; chunk c + 2's may still be in flight
    C3C_VMCNT(KTG * WCO + 2 * NR);
    barrier();
  };

  // prologue: chunks 0 and 1 into buffers and weight sets 0 and 1, slot 0
  // of chunk 0 pre-read
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  load_w(0, w[0]);
  stage_act(0, lds0);
  load_w(1, w[1]);
  stage_act(1, lds1);
  C3C_VMCNT(KTG * WCO + 2 * NR);
  barrier();
  read_a(lds0, 0, avs[0], 0u);

  // three stages a round: buffers and weight sets 0, 1, 2 in turn (stages
  // past the last chunk read zeros: zero-size sources, out-of-range weights;
  // a round with early exits made the register allocator copy the
  // accumulators between the stage copies)
  for (int c = 0; c < a.chunks; c += 3) {
    stage(c, I0{});
    stage(c + 1, I1{});
    stage(c + 2, I2{});
  }
#undef C3C_VMCNT

  // epilogue: lane l holds pixels 4 (l / 16) .. + 3 of output channel l % 16
  // of each fragment; bias once, one round-to-nearest-even, NCTHW store
  uint16_t* ybase = a.y + static_cast<int64_t>(n) * a.Co * a.To * a.hw;
#pragma unroll
  for (int cf = 0; cf < WCO; ++cf) {
    const int co = ctile * TCO + wv * 16 * WCO + cf * 16 + (lane & 15);
    if (co >= a.Co) continue;
    const float bb = bias_v[cf];
    uint16_t* yrow = ybase + static_cast<int64_t>(co) * a.To * a.hw;
#pragma unroll
    for (int pf = 0; pf < NPF; ++pf) {
      const int p = px0 + pf * 16 + 4 * g;
      if (p >= a.hw) continue;
      const uint32_t v01 = __builtin_bit_cast(
          uint32_t, __builtin_convertvector((f32x2{acc[cf][pf][0] + bb, acc[cf][pf][1] + bb}), bf16x2));
      const uint32_t v23 = __builtin_bit_cast(
          uint32_t, __builtin_convertvector((f32x2{acc[cf][pf][2] + bb, acc[cf][pf][3] + bb}), bf16x2));
      *reinterpret_cast<uint2*>(yrow + p) = make_uint2(v01, v23);
    }
  }
}

bool aligned_to(const void* p, uintptr_t m) { return (reinterpret_cast<uintptr_t>(p) & (m - 1)) == 0; }

}  // namespace

bool tap1x1_eligible(const Geo& g, const void* x, const void* cache, const void* y) {
  const c3c_conv_desc& d = g.d;
  // buffer offsets are 32-bit: one 32-channel stage slab and the packed weights must fit
  const int64_t frames = d.T > d.Tc ? d.T : d.Tc;
  if (static_cast<int64_t>(TK) * frames * d.H * d.W * 2 >= 0x7fffffff ||
      pack_dims(d).elems() * 2 >= 0x7fffffff)
    return false;
  return (d.H * d.W) % 8 == 0 && aligned_to(x, 16) && (cache == nullptr || aligned_to(cache, 16)) &&
         aligned_to(y, 8);
}

int64_t tap1x1_blocks(const Geo& g) {
  return (g.d.H * g.d.W + TPX - 1) / TPX * ((g.d.Co + TCO - 1) / TCO) * g.To * g.d.N;
}

namespace {

// Whether every frame of the new cache is read by some output frame
// (f = t s_t + k d_t - p_l with t < To, k < Kt), so that the kernels, which
// copy a cache frame when they stage it, write the whole new cache.
bool stages_new_cache(const Geo& g) {
  const c3c_conv_desc& d = g.d;
  for (int64_t f = g.Z - g.L; f < g.Z; ++f) {
    bool found = false;
    for (int64_t k = 0; k < d.Kt && !found; ++k) {
      const int64_t kd = f + g.p_l - k * d.dil_t;
      found = kd >= 0 && kd % d.stride_t == 0 && kd / d.stride_t < g.To;
    }
    if (!found) return false;
  }
  return true;
}

}  // namespace

hipError_t launch_tap1x1(const Geo& g, const void* x, const void* cache, const void* wpack,
                         const void* bias, void* y, void* cache_out, bool* cache_written,
                         hipStream_t s, LaunchInfo* info) {
  const c3c_conv_desc& d = g.d;
  const PackDims p = pack_dims(d);
  if (cache_written) *cache_written = false;
  if (!tap1x1_eligible(g, x, cache, y)) return hipErrorInvalidValue;
  TapArgs a;
  a.x = static_cast<const uint16_t*>(x);
  a.cache = static_cast<const uint16_t*>(cache);
  a.wpack = static_cast<const u32x4*>(wpack);
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
  a.chunks = static_cast<int>(p.chunks);
  a.cofrags = static_cast<int>(p.cofrags);
  a.px_tiles = static_cast<int>((a.hw + TPX - 1) / TPX);
  a.co_tiles = static_cast<int>((d.Co + TCO - 1) / TCO);
  a.wpack_bytes = static_cast<uint32_t>(p.elems() * 2);
  a.has_bias = d.has_bias ? 1 : 0;
  a.cache_out = static_cast<uint16_t*>(cache_out);
  a.L = static_cast<int>(g.L);
  a.write_cache = 0;
  // the chunk-stage form for one output frame (Kt <= 3), else one stage per
  // tap and chunk
  // (its source offsets span every channel of a frame, three chunks past the
  // last included, and its new-cache offsets every channel and frame, in 32
  // bits)
  const bool chunk_form = g.To == 1 && d.Kt <= KTG &&
                          (d.Ci + 3 * TK) * (d.T + d.Tc) * d.H * d.W * 2 < 0x7fffffff;
  // the new cache from the staged tiles when every frame of it is staged
  // (32-bit offsets within a 32-channel slab of it; a tap mask of 32 bits)
  a.write_cache = g.L > 0 && cache_out != nullptr && aligned_to(cache_out, 16) && d.Kt <= 32 &&
                  static_cast<int64_t>(TK) * g.L * a.hw * 2 < 0x7fffffff && stages_new_cache(g);
  const int64_t blocks = tap1x1_blocks(g);
  if (info) {
    info->kernel = C3C_KERNEL_TAP1X1;
    info->tile_co = TCO;
    info->tile_h = 0;
    info->tile_w = TPX;
    info->workgroups = blocks;
    info->cache_in_kernel = a.write_cache != 0;
    if (cache_written) *cache_written = a.write_cache != 0;
    return hipSuccess;
  }
  if (cache_written) *cache_written = a.write_cache != 0;
  if (blocks == 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  a.nblocks = static_cast<int>(blocks);
  const dim3 grid(static_cast<unsigned>(blocks)), block(256);
  if (chunk_form)
    hipLaunchKernelGGL(conv_tap1x1_chunk, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(conv_tap1x1, grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace c3c
