// Fast route, bf16, 3x3 spatial kernel with few output channels (Co <= 5,
// e.g. a decoder's RGB head): the spatial taps go to the matrix cores' N
// dimension instead of K.
//
// Output frame o of batch element n is (Eq. 2, active taps of Eq. 4)
//   y[co][h][w] = b[co] + sum_{k active} sum_{i,j} sum_ci w[co][ci][k][i][j] z[ci][f_k][h+i-1][w+j-1].
// Writing D[p][(i,j,co)] = sum_k sum_ci w[co][ci][k][i][j] z[ci][f_k][p] for every
// input position p, this is y[co][h][w] = b[co] + sum_{i,j} D[(h+i-1, w+j-1)][(i,j,co)]
// (D is 0 outside the image, as the zero padding of z makes it).  D is a
// 1x1 product with 9 Co columns: 27 for Co = 3, two 16-wide fragments of
// v_mfma_f32_16x16x32_bf16, where the 3x3 kernel would pad Co = 3 to 16 for
// each of the 9 spatial taps.
//
// Workgroup = 6 output rows x 48 output columns of one spatial tile, for
// every output frame: the output frames are taken in groups of OG (4, or 2
// with three column fragments), and a group stages each source frame f it
// needs (f = o + k d_t - p_l for its frames o and the taps k, inside Z)
// once per 32-channel chunk, from an input window of 8 rows x 64 columns
// (origin one row above and eight columns left of the output tile, so that
// every 16-byte row segment of the window is aligned).  A staged (frame,
// chunk) feeds every output frame of the group that reads it, each with its
// own tap's weights, into that frame's accumulators: a source frame is read
// once per group instead of once per output frame that uses it.  4 waves,
// wave v owning window rows 2v, 2v + 1: 8 pixel fragments x NF column
// fragments per output frame of the group (up to 256 accumulator registers,
// one workgroup per compute unit).
// Staging: a stage's [32 ch][512 px] window tile goes from memory straight
// into LDS (buffer loads with the LDS destination, 16 bytes a lane, no
// registers): one load instruction of a wave fills one channel's 8 x 64
// window, lane l taking window row l / 8, columns 8 (l % 8) .. + 7 (zeros
// outside the image or past the last channel).  It is read back with the
// transposing ds_read_b64_tr_b16 (the A operand: 8 channels of one pixel per
// lane).  The B operand for column n = 9-tap index ij times Co plus co is
// the 16-byte lane slot of the packed 3x3 weights' fragment (tap k*9 + ij,
// chunk, 0) that holds output channel co (the fast route's one weight
// packing serves this kernel too); every wave needs the same B operands, so
// the workgroup gathers them once, at its start, into an LDS table of 1 KiB
// lane-ordered entries (temporal tap k, chunk, column fragment q), and a
// stage reads its B operands from there: a stage's only vector-memory loads
// are its window's 32 (one per channel; on these loads the texture
// addresser, not HBM, sets the pace).
// Pipeline: NB = 4 (or 3, when the table needs the room) LDS buffers; during
// stage s the waves issue stage s + NB - 1's window loads into buffer
// (s + NB - 1) % NB (last read in stage s - 1), run stage s's products from
// buffer s % NB, then wait for their own loads of stage s + 1 and meet at
// one plain barrier, so the later stages' loads stay in flight across it.
// The stage count is padded to a multiple of NB with stages that read zeros
// and skip their products.  Per stage the scalar work is a few additions:
// the source pointer and the table offsets step by one chunk, and only a
// new source frame recomputes them (with the tap of each output frame).
// After a group's last stage, its output frames' accumulators go to LDS as
// D[n][px] in fp32, NB / NF frames at a time (one stage buffer per column
// fragment), and the workgroup sums the nine shifted D values of each
// output, adds the bias once and rounds once.
// A frame of the new cache is copied out of the stage buffer by the group
// that first stages it (its interior segments: each element has one
// writer), so the caller copies no cache when every cache frame is staged.
//
// Requires W a multiple of 8, 16-byte-aligned x / cache, 8-byte-aligned y
// (and a 16-byte-aligned cache_out for the fused cache write).
#include <algorithm>
#include <type_traits>

#include "c3c_internal.h"

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
typedef __attribute__((address_space(3))) void lds_void;

constexpr int HK = 32;                 // input channels per stage
constexpr int HR = 8, HC = 64;         // input window rows x columns
constexpr int OR = 6, OC = 48;         // output rows x columns per workgroup
constexpr int HPX = HR * HC;           // window pixels
constexpr int HPF = 2 * (HC / 16);     // pixel fragments per wave (2 rows)
constexpr int HSEG = HK * HPX / 8;     // 16-byte segments of a stage tile
static_assert(HSEG == 256 * 8 && HR * HC / 8 == 64,
              "a wave stages 8 channels, one 64-segment window per load instruction");
// LDS offset of staged channel row c: 1024 B + 32 B, and 128 B more after
// every 8 channels.  The 32 lanes one transposing read serves per cycle take
// 32 B from each of channels {0..3, 8..11} (+4, +16, +20 for the other
// halves): banks 0, 8, 16, 24 and 32, 40, 48, 56, disjoint 8-bank groups.
constexpr int HPITCH = HPX * 2 + 32;
constexpr int hrow(int c) { return c * HPITCH + (c >> 3) * 128; }
constexpr int HBUF = hrow(HK);
constexpr int kLdsBytes = 160 * 1024;  // LDS of a compute unit
constexpr int max_co(int nf) { return 16 * nf / 9; }
// the weight table beside NB stage buffers: bytes, and 1 KiB entries
constexpr int wtab_bytes(int nb) { return (kLdsBytes - nb * HBUF - (nb == 4 ? 0 : 16)) / 1024 * 1024; }
constexpr int wtab_entries(int nb) { return wtab_bytes(nb) / 1024; }
int head_table_entries(const c3c_conv_desc& d) {
  return static_cast<int>(d.Kt * ((d.Ci + HK - 1) / HK) * ((9 * d.Co + 15) / 16));
}
// D rows (one per column n) of the window's 512 pixels, 516 floats apart: the
// 16 lanes of a fragment row write 16 consecutive n with 16-byte stores, and
// 516 = 4 mod 64 banks puts them in 16 disjoint 4-bank groups; the 16 rows of
// one column fragment fill one stage buffer
constexpr int DPITCH = HPX + 4;
static_assert(16 * DPITCH * 4 <= HBUF, "a column fragment of D fits one stage buffer");

struct HeadArgs {
  const uint16_t* x;
  const uint16_t* cache;
  const u32x4* wpack;
  const uint16_t* bias;
  uint16_t* y;
  uint16_t* cache_out;
  int64_t hw;
  int N, Ci, Co, T, Tc, H, W, To, Z, dt, p_l, Kt, L;
  int chunks, cofrags, tiles_w, tiles_h, nblocks;
  uint32_t wpack_bytes;
  int has_bias, write_cache;
};

template <int V>
using IC = std::integral_constant<int, V>;

// OG output frames per pass (a group); NF 16-column fragments of D per tap;
// NB stage buffers.
template <int NF, int OG, int NB>
__global__ __launch_bounds__(256, 1) void conv_head(HeadArgs a) {
  static_assert(NF <= NB && (NB == 3 || NB == 4), "D's column fragments go one per stage buffer");
  constexpr int AHEAD = NB - 1;  // stages between a window load and its use
  // the stage buffers and the weight table, each its own array: the
  // compiler then knows that a load into one does not write what is read
  // from another
  __shared__ __align__(16) unsigned char lds0[HBUF];
  __shared__ __align__(16) unsigned char lds1[HBUF];
  __shared__ __align__(16) unsigned char lds2[HBUF];
  __shared__ __align__(16) unsigned char lds3[NB == 4 ? HBUF : 16];
  __shared__ __align__(16) unsigned char wtab[wtab_bytes(NB)];
  auto bufp = [&](int q) -> unsigned char* { return q == 0 ? lds0 : q == 1 ? lds1 : q == 2 ? lds2 : lds3; };
  constexpr uint32_t OOB = 0x80000000u;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // the bias of every output channel (Co <= 5), loaded at the start: loaded
  // in the gather loop, each load's wait also waited for the stores before
  // it (no bias, or a channel past Co: an out-of-range offset, 0)
  float bias_c[5];
  {
    const __amdgpu_buffer_rsrc_t brs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(a.bias), 0, a.has_bias ? a.Co * 2 : 0, 0x00020000);
#pragma unroll
    for (int c = 0; c < 5; ++c)
      bias_c[c] = __uint_as_float(static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b16(brs, 2u * c, 0, 0)) << 16);
  }

  // workgroups numbered so that each XCD runs a contiguous range of
  // neighbouring spatial tiles (their windows overlap in the halo rows)
  int b;
  {
    const int per = a.nblocks / 8, rem = a.nblocks % 8;
    const int xcd = static_cast<int>(blockIdx.x) % 8, slot = static_cast<int>(blockIdx.x) / 8;
    b = (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + slot;
  }
  const int tw = b % a.tiles_w;
  b /= a.tiles_w;
  const int th = b % a.tiles_h;
  const int n = b / a.tiles_h;
  const int h0 = th * OR, w0 = tw * OC;
  const int wh0 = h0 - 1, ww0 = w0 - 8;  // window origin

  // this lane's window segment (row lane / 8, columns 8 (lane % 8) .. + 7),
  // staged for channels 8 wave .. + 7 of each stage; outside the image an
  // out-of-range offset (zeros; W is a multiple of 8, so a segment is wholly
  // inside or outside).  s_in: the segment lies in this tile's output rows
  // and columns (the part of the window the new cache takes from here)
  const int sr = lane >> 3, ssg = lane & 7;
  const int gh = wh0 + sr, gw = ww0 + 8 * ssg;
  const bool s_ok = gh >= 0 && gh < a.H && gw >= 0 && gw < a.W;
  const uint32_t s_px = s_ok ? static_cast<uint32_t>(gh * a.W + gw) * 2u : OOB;
  const bool s_in = s_ok && sr >= 1 && sr <= OR && ssg >= 1 && ssg <= OC / 8;
  const int ch0 = 8 * wave;                                  // first staged channel
  const uint32_t lrow = static_cast<uint32_t>(hrow(8) * wave);  // its LDS row

  // weight table: entry e = (k chunks + c) NF + q holds, for lane l, the B
  // operand of column n = 16 q + l % 16 = (ij = n / Co, co = n % Co), for
  // n < 9 Co: the lane slot co + 16 (l / 16) of packed fragment (tap
  // k 9 + ij, chunk c, output fragment 0).  Columns past 9 Co take tap
  // (0, 0)'s slot: their D is never read.
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<u32x4*>(a.wpack), 0, static_cast<int>(a.wpack_bytes), 0x00020000);
  const uint32_t frag_bytes = static_cast<uint32_t>(a.cofrags) * 1024u;
  uint32_t w_off[NF];
#pragma unroll
  for (int q = 0; q < NF; ++q) {
    const int col = 16 * q + (lane & 15);
    const bool used = col < 9 * a.Co;
    const int ij = used ? col / a.Co : 0, co = used ? col % a.Co : 0;
    w_off[q] = static_cast<uint32_t>(ij * a.chunks) * frag_bytes +
               static_cast<uint32_t>(co + 16 * (lane >> 4)) * 16u;
  }

  // transposing operand read of pixel fragment pf of this wave (window row
  // 2 wave + pf / (HC / 16), columns 16 (pf % (HC / 16)) ..): lane j of 16-lane block g names
  // channel 8g + 4h + j / 4 at pixel group 4 (j % 4)
  const int j = lane & 15, g = lane >> 4;
  const int ra = hrow(8 * g + (j >> 2)) + (2 * wave * HC + 4 * (j & 3)) * 2;
  auto read_a = [&](const unsigned char* L, int pf) __attribute__((always_inline)) {
    const unsigned char* p = L + ra + ((pf / (HC / 16)) * HC + (pf % (HC / 16)) * 16) * 2;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 4 * HPITCH));
    return i16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  };

  f32x4 acc[OG][NF][HPF];
  const int64_t plane = static_cast<int64_t>(a.To) * a.hw;
  const int64_t cs_c = static_cast<int64_t>(a.Tc) * a.hw, cs_x = static_cast<int64_t>(a.T) * a.hw;
  const int64_t cl = static_cast<int64_t>(a.L) * a.hw;
  const uint32_t ccs = static_cast<uint32_t>(cl * 2);  // bytes between new-cache channel planes
  int f_done = -1;  // the last source frame staged by an earlier group

  // wait until at most n vector-memory operations of this wave are
  // outstanding (the LDS and export counters left alone)
#define C3C_VMCNT(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | (7 << 4) | (15 << 8))
  auto barrier = [] { asm volatile("s_barrier" ::: "memory"); };

  for (int og0 = 0; og0 < a.To; og0 += OG) {
    // Source frames of this group's output frames [og0, og0 + OG): the
    // frames f = o + k dt - p_l inside Z (Eq. 4), each staged once per
    // 32-channel chunk; stage (f, c) feeds every output frame o of the group
    // with o = f + p_l - k dt for some tap k.
    const int og1 = og0 + OG < a.To ? og0 + OG : a.To;
    const int f_lo = og0 - a.p_l > 0 ? og0 - a.p_l : 0;
    const int f_top = og1 - 1 + (a.Kt - 1) * a.dt - a.p_l;
    const int f_hi = f_top < a.Z - 1 ? f_top : a.Z - 1;
    const int nst = f_hi >= f_lo ? (f_hi - f_lo + 1) * a.chunks : 0;
    const int padded = (nst + NB - 1) / NB * NB;

#pragma unroll
    for (int u = 0; u < OG; ++u)
#pragma unroll
      for (int q = 0; q < NF; ++q)
#pragma unroll
        for (int pf = 0; pf < HPF; ++pf) acc[u][q][pf] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Stages run frame by frame, chunk by chunk, from (f_lo, 0); frames past
    // f_hi are padding.  Two cursors: the window loads and the stage being
    // computed.
    // window cursor: frame af, chunk ac; ap = channel 32 ac of frame af
    int af = f_lo, ac = 0;
    const uint16_t* ap = a.x;
    uint32_t acs = 0;     // bytes between the source's channel planes
    int64_t astep = 0;    // elements between consecutive chunks
    auto act_frame = [&]() __attribute__((always_inline)) {
      const bool in_cache = af < a.Tc;
      const int64_t cstride = in_cache ? cs_c : cs_x;
      ap = af <= f_hi ? (in_cache ? a.cache + static_cast<int64_t>(af) * a.hw
                                  : a.x + static_cast<int64_t>(af - a.Tc) * a.hw) +
                            static_cast<int64_t>(n) * a.Ci * cstride
                      : a.x;
      acs = static_cast<uint32_t>(cstride * 2);
      astep = HK * cstride;
    };
    // the window loads of the cursor's stage into buffer L; the source is
    // bounded after the chunk's last real channel (channels past Ci read 0),
    // empty past the last frame
    auto issue_act = [&](unsigned char* L) __attribute__((always_inline)) {
      const int c0 = ac * HK;
      const uint32_t bytes = af <= f_hi ? static_cast<uint32_t>(min(HK, a.Ci - c0) - 1) * acs +
                                              static_cast<uint32_t>(a.hw) * 2u
                                        : 0u;
      const __amdgpu_buffer_rsrc_t rs =
          __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(ap), 0, static_cast<int>(bytes), 0x00020000);
#pragma unroll
      for (int i = 0; i < 8; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)(L + lrow + i * HPITCH), 16,
                                                 s_px + static_cast<uint32_t>(ch0 + i) * acs, 0, 0, 0);
      if (++ac == a.chunks) {
        ac = 0;
        ++af;
        act_frame();
      } else {
        ap += astep;
      }
    };
    // compute cursor: frame cf, chunk cc; per output frame u of the group
    // the table offset of its tap's entries (tap k = (f + p_l - o) / d_t
    // when that is a whole tap index; otherwise its products are skipped:
    // bit u of wok clear, offset 0)
    int cf = f_lo, cc = 0;
    uint32_t wb[OG], wok = 0;
    auto c_frame = [&]() __attribute__((always_inline)) {
      wok = 0;
#pragma unroll
      for (int u = 0; u < OG; ++u) {
        const int o = og0 + u, kd = cf + a.p_l - o;
        const int k = kd >= 0 ? kd / a.dt : -1;
        const bool ok = cf <= f_hi && o < og1 && kd >= 0 && kd % a.dt == 0 && k < a.Kt;
        wb[u] = ok ? static_cast<uint32_t>(k * a.chunks * NF) * 1024u : 0u;
        wok |= (ok ? 1u : 0u) << u;
      }
    };
    auto c_next = [&]() __attribute__((always_inline)) {
      if (++cc == a.chunks) {
        cc = 0;
        ++cf;
        c_frame();
      } else {
#pragma unroll
        for (int u = 0; u < OG; ++u) wb[u] += (wok >> u) & 1u ? NF * 1024u : 0u;
      }
    };
    // A frame of the new cache staged for the first time (workgroup-uniform)
    // has its interior segments copied from the stage buffer to cache_out,
    // through a resource that ends after the chunk's last real channel.
    // Returns whether it stored (8 stores a lane).
    auto copy_cache = [&](const unsigned char* L) __attribute__((always_inline)) {
      const bool on = a.write_cache && cf <= f_hi && cf > f_done && cf >= a.Z - a.L;
      if (on) {
        const int c0 = cc * HK;
        const uint32_t cbytes = static_cast<uint32_t>(min(HK, a.Ci - c0) - 1) * ccs + static_cast<uint32_t>(a.hw) * 2u;
        const __amdgpu_buffer_rsrc_t crs = __builtin_amdgcn_make_buffer_rsrc(
            a.cache_out + (static_cast<int64_t>(n) * a.Ci + c0) * cl + static_cast<int64_t>(cf - (a.Z - a.L)) * a.hw,
            0, static_cast<int>(cbytes), 0x00020000);
        u32x4 v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = *reinterpret_cast<const u32x4*>(L + lrow + i * HPITCH + lane * 16);
#pragma unroll
        for (int i = 0; i < 8; ++i)
          __builtin_amdgcn_raw_buffer_store_b128(v[i], crs, s_in ? static_cast<uint32_t>(ch0 + i) * ccs + s_px : OOB,
                                                 0, 0);
      }
      return on;
    };

    // one stage from buffer B: the cache copy, the window loads of stage
    // s + NB - 1 into buffer (B + NB - 1) % NB, the B operands from the
    // table and the products of every output frame the stage feeds, then
    // this wave's loads of stage s + 1 awaited and one barrier.  After those
    // loads the wave issued, in each of its last NB - 2 stages, 8 stores if
    // it copied cache and 8 window loads; sth has a bit per such stage that
    // stored, so the wait is exact and later loads stay in flight.
    uint32_t sth = 0;
    constexpr uint32_t sth_mask = NB == 4 ? 3u : 1u;
    auto stage = [&](auto B) __attribute__((always_inline)) {
      constexpr int b0 = decltype(B)::value, bn = (b0 + AHEAD) % NB;
      const unsigned char* cur = bufp(b0);
      sth = ((sth << 1) | (copy_cache(cur) ? 1u : 0u)) & sth_mask;
      issue_act(bufp(bn));
      u32x4 bv[OG][NF];
#pragma unroll
      for (int u = 0; u < OG; ++u)
#pragma unroll
        for (int q = 0; q < NF; ++q)
          bv[u][q] = *reinterpret_cast<const u32x4*>(wtab + wb[u] + q * 1024 + lane * 16);
      i16x8 av[HPF];
#pragma unroll
      for (int pf = 0; pf < HPF; ++pf) av[pf] = read_a(cur, pf);
#pragma unroll
      for (int u = 0; u < OG; ++u) {
        if (!((wok >> u) & 1u)) continue;  // workgroup-uniform
#pragma unroll
        for (int pf = 0; pf < HPF; ++pf)
#pragma unroll
          for (int q = 0; q < NF; ++q)
            acc[u][q][pf] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, av[pf]), __builtin_bit_cast(bf16x8, bv[u][q]), acc[u][q][pf], 0, 0, 0);
      }
      c_next();
      if (sth == 0)
        C3C_VMCNT((AHEAD - 1) * 8);
      else if (sth == 3)
        C3C_VMCNT((AHEAD - 1) * 8 + 16);
      else
        C3C_VMCNT((AHEAD - 1) * 8 + 8);
      barrier();
    };

    // prologue: the weight table (first group only), then stages
    // 0 .. NB - 2 into buffers 0 .. NB - 2
    if (og0 == 0) {
      const int nent = a.Kt * a.chunks * NF;
      for (int e = wave; e < nent; e += 4) {
        const int q = e % NF, kc = e / NF;
        const uint32_t base = static_cast<uint32_t>((kc / a.chunks) * 9 * a.chunks + kc % a.chunks) * frag_bytes;
        const uint32_t vo = base + w_off[q];  // (a named offset: the host pass drops the kernel
                                              // when this builtin's argument indexes w_off)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(wrs, (lds_void*)(wtab + e * 1024), 16, vo, 0, 0, 0);
      }
    }
    act_frame();
    c_frame();
    issue_act(lds0);
    issue_act(lds1);
    if constexpr (NB == 4) issue_act(lds2);
    C3C_VMCNT((AHEAD - 1) * 8);  // the table and stage 0 have landed
    barrier();
    for (int s = 0; s < padded; s += NB) {
      stage(IC<0>{});
      stage(IC<1>{});
      stage(IC<2>{});
      if constexpr (NB == 4) stage(IC<3>{});
    }
    // the loads issued past the last stage (zeros) land before LDS is reused
    C3C_VMCNT(0);
    barrier();
    f_done = f_hi;

    // per batch of FB output frames of the group: D[n][window pixel] in
    // fp32, column fragment q of the batch's frame du in stage buffer
    // NF du + q (lane l holds pixels 4 (l / 16) .. + 3 of column
    // 16 q + l % 16 of each fragment), then the gather: output (co, row r,
    // columns 4 c4 .. + 3) sums D[(i j) Co + co] at window row r + i, window
    // columns 7 + 4 c4 + j .. + 3; bias once, one round-to-nearest-even,
    // 8-byte NCTHW store
    constexpr int FB = NB / NF;  // output frames per batch
    constexpr int ITEMS = OR * (OC / 4);  // 4-column output groups per (frame, co)
#pragma unroll
    for (int u0 = 0; u0 < OG; u0 += FB) {
      if (og0 + u0 >= og1) break;
#pragma unroll
      for (int du = 0; du < FB && u0 + du < OG; ++du) {
        if (og0 + u0 + du >= og1) break;
#pragma unroll
        for (int q = 0; q < NF; ++q) {
          if (16 * q + (lane & 15) >= 9 * a.Co) continue;
          float* Dq = reinterpret_cast<float*>(bufp(NF * du + q)) + (lane & 15) * DPITCH;
#pragma unroll
          for (int pf = 0; pf < HPF; ++pf) {
            const int px = (2 * wave + pf / (HC / 16)) * HC + (pf % (HC / 16)) * 16 + 4 * g;
            *reinterpret_cast<f32x4*>(Dq + px) = acc[u0 + du][q][pf];
          }
        }
      }
      __syncthreads();
      const int nfr = min(FB, og1 - og0 - u0);
      for (int t = tid; t < nfr * a.Co * ITEMS; t += 256) {
        const int du = t / (a.Co * ITEMS), t2 = t % (a.Co * ITEMS);
        const int co = t2 / ITEMS, rem = t2 % ITEMS;
        const int r = rem / (OC / 4), c4 = rem % (OC / 4);
        const int h = h0 + r, w = w0 + 4 * c4, o = og0 + u0 + du;
        if (h >= a.H || w >= a.W) continue;
        const float bb = co == 0 ? bias_c[0] : co == 1 ? bias_c[1] : co == 2 ? bias_c[2] : co == 3 ? bias_c[3] : bias_c[4];
        float s4[4] = {bb, bb, bb, bb};
#pragma unroll
        for (int i = 0; i < 3; ++i)
#pragma unroll
          for (int jj = 0; jj < 3; ++jj) {
            const int col = (i * 3 + jj) * a.Co + co;
            const float* src = reinterpret_cast<const float*>(bufp(NF * du + (col >> 4))) + (col & 15) * DPITCH +
                               (r + i) * HC + 7 + 4 * c4 + jj;
#pragma unroll
            for (int e = 0; e < 4; ++e) s4[e] += src[e];
          }
        const uint32_t v01 = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{s4[0], s4[1]}), bf16x2));
        const uint32_t v23 = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{s4[2], s4[3]}), bf16x2));
        uint16_t* dst = a.y + (static_cast<int64_t>(n) * a.Co + co) * plane + static_cast<int64_t>(o) * a.hw +
                        static_cast<int64_t>(h) * a.W + w;
        *reinterpret_cast<uint2*>(dst) = make_uint2(v01, v23);
      }
      __syncthreads();  // D is rewritten by the next batch, the stage buffers by the next group
    }
  }
#undef C3C_VMCNT
}

bool aligned_to(const void* p, uintptr_t m) { return (reinterpret_cast<uintptr_t>(p) & (m - 1)) == 0; }

}  // namespace

bool head_eligible(const Geo& g, const void* x, const void* cache, const void* y) {
  const c3c_conv_desc& d = g.d;
  // the weight table must fit beside three stage buffers
  if (d.Co > max_co(3) || d.W % 8 != 0 || head_table_entries(d) > wtab_entries(3)) return false;
  // buffer offsets are 32-bit: one 32-channel slab of a source frame and the
  // packed weights must fit
  const int64_t frames = d.T > d.Tc ? d.T : d.Tc;
  if (static_cast<int64_t>(HK) * frames * d.H * d.W * 2 >= 0x7fffffff ||
      pack_dims(d).elems() * 2 >= 0x7fffffff)
    return false;
  return aligned_to(x, 16) && (cache == nullptr || aligned_to(cache, 16)) && aligned_to(y, 8);
}

hipError_t launch_head(const Geo& g, const void* x, const void* cache, const void* wpack,
                       const void* bias, void* y, void* cache_out, bool* cache_written,
                       hipStream_t s, LaunchInfo* info) {
  const c3c_conv_desc& d = g.d;
  if (!head_eligible(g, x, cache, y)) return hipErrorInvalidValue;
  const PackDims p = pack_dims(d);
  HeadArgs a;
  a.x = static_cast<const uint16_t*>(x);
  a.cache = static_cast<const uint16_t*>(cache);
  a.wpack = static_cast<const u32x4*>(wpack);
  a.bias = static_cast<const uint16_t*>(bias);
  a.y = static_cast<uint16_t*>(y);
  a.cache_out = static_cast<uint16_t*>(cache_out);
  a.hw = d.H * d.W;
  a.N = static_cast<int>(d.N);
  a.Ci = static_cast<int>(d.Ci);
  a.Co = static_cast<int>(d.Co);
  a.T = static_cast<int>(d.T);
  a.Tc = static_cast<int>(d.Tc);
  a.H = static_cast<int>(d.H);
  a.W = static_cast<int>(d.W);
  a.To = static_cast<int>(g.To);
  a.Z = static_cast<int>(g.Z);
  a.dt = static_cast<int>(d.dil_t);
  a.p_l = static_cast<int>(g.p_l);
  a.Kt = static_cast<int>(d.Kt);
  a.chunks = static_cast<int>(p.chunks);
  a.cofrags = static_cast<int>(p.cofrags);
  a.tiles_w = static_cast<int>((d.W + OC - 1) / OC);
  a.tiles_h = static_cast<int>((d.H + OR - 1) / OR);
  a.wpack_bytes = static_cast<uint32_t>(p.elems() * 2);
  a.has_bias = d.has_bias ? 1 : 0;
  a.L = static_cast<int>(g.L);
  // The kernel stages every frame in [max(0, -p_l), min(Z - 1, To - 1 +
  // (Kt - 1) d_t - p_l)] once per spatial tile and writes the new cache's
  // frames among them (interior segments, one writer per element); a cache
  // frame outside that range falls to the caller's copy.  Cache frames are
  // also L2-resident 32-channel slabs, so the same 32-bit offset limit holds.
  const int64_t f_first = g.p_l < 0 ? -g.p_l : 0;
  const int64_t f_last = std::min<int64_t>(g.Z - 1, g.To - 1 + (d.Kt - 1) * d.dil_t - g.p_l);
  a.write_cache = (g.L > 0 && cache_out != nullptr && g.Z - g.L >= f_first && g.Z - 1 <= f_last &&
                   static_cast<int64_t>(HK) * g.L * a.hw * 2 < 0x7fffffff &&
                   aligned_to(cache_out, 16)) ? 1 : 0;
  if (cache_written) *cache_written = a.write_cache != 0;
  const int64_t blocks = static_cast<int64_t>(a.tiles_w) * a.tiles_h * d.N;
  if (info) {
    info->kernel = C3C_KERNEL_HEAD;
    info->tile_co = d.Co;
    info->tile_h = OR;
    info->tile_w = OC;
    info->workgroups = blocks;
    info->cache_in_kernel = a.write_cache != 0;
    return hipSuccess;
  }
  if (blocks == 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  a.nblocks = static_cast<int>(blocks);
  const int nf = static_cast<int>((9 * d.Co + 15) / 16);
  const bool nb4 = head_table_entries(d) <= wtab_entries(4);
  const dim3 grid(static_cast<unsigned>(blocks)), block(256);
  // output frames per group: 4 (the 256 accumulator registers of 4 frames x
  // 2 fragments x 8 pixel fragments), 2 with three column fragments; four
  // stage buffers when the weight table fits beside them, else three
  if (nf == 1 && nb4)
    hipLaunchKernelGGL((conv_head<1, 4, 4>), grid, block, 0, s, a);
  else if (nf == 1)
    hipLaunchKernelGGL((conv_head<1, 4, 3>), grid, block, 0, s, a);
  else if (nf == 2 && nb4)
    hipLaunchKernelGGL((conv_head<2, 4, 4>), grid, block, 0, s, a);
  else if (nf == 2)
    hipLaunchKernelGGL((conv_head<2, 4, 3>), grid, block, 0, s, a);
  else if (nb4)
    hipLaunchKernelGGL((conv_head<3, 2, 4>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((conv_head<3, 2, 3>), grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace c3c
