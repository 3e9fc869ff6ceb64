// bf16 fast route: the cache-aware lowering of one cached causal Conv3D call
// (paper Sec. 4, Eq. 2 and Eq. 4, Alg. 1) as ONE implicit-GEMM kernel on
// gfx950 bf16 matrix cores, with the bias and the cache update fused in.
//
// Mapping of the paper's procedure
//   * Alg. 1 folds the valid frames [z_l, z_h) of tap k into the batch and
//     runs one Conv2D per active tap into an accumulator A.  Here a workgroup
//     owns one output frame o (plus a spatial tile and an output-channel
//     tile); the taps k active for o (Eq. 4: o_l(k) <= o < o_h(k)) read source
//     frame o + delta_k directly from the cache or the new chunk -- the fold
//     and the concatenation [C; X] are index maps, never copies -- and all
//     taps accumulate into the same fp32 registers.
//   * The bias is added once, in the epilogue, before one round-to-nearest-
//     even conversion to bf16; the output is stored NCTHW.
//   * The cache update (the last L frames of Z) is written by the workgroup
//     that stages each of those frames for its last tap, from the registers
//     the frame was loaded into, so it costs no extra read.
//
// GEMM view per output frame: D[co][px] = sum_K Wk[co][K] * Z[K][px], K =
// (kt, kh, kw, ci).  The matrix-core instruction is v_mfma_f32_16x16x32_bf16
// computing D^T[px][co]: A = activations (16 pixels x 32 input channels),
// B = weights (32 input channels x 16 output channels), C/D = 16 x 16 fp32,
// lane l holding pixels 4*(l/16) .. +3 of output channel l % 16 -- four
// consecutive output pixels, stored with one 8-byte write.
//
// Data movement
//   * Weights (B operand) come pre-packed in fragment order
//     (c3c_weight_repack): one 16-byte load per lane per fragment, straight
//     from L2 into registers, two (kh, kw) steps ahead of their use (a
//     3-slot register ring).
//   * Activations (A operand) are staged per (tap, 32-channel chunk) as a
//     halo tile [BH+2][BW+2][32 ch] in LDS, channel-innermost with a 96-byte
//     pixel pitch (bank-conflict-free for the operand reads), so that each
//     lane reads its 8 K-consecutive channels with one ds_read_b128 and the
//     nine (kh, kw) offsets of the 3x3 kernel are nine immediate address
//     offsets into the same tile.  Global reads are 16-byte row segments of
//     the NCTHW planes; an 8x8 register transpose (v_perm) turns 8 channel
//     rows x 8 pixels into 8 pixel records.  Tiles rotate through NBUF LDS
//     buffers: the next stage's global loads are in flight while the current
//     stage computes, and each operand fragment is re-read from LDS right
//     after its last use (one register set, no double buffer).
//   * Workgroups are numbered so that each of the 8 XCDs (which take
//     workgroups round-robin) runs a contiguous range of tiles -- consecutive
//     output frames of the same spatial tile, then neighbouring tiles -- so
//     the frames shared by neighbouring taps and the halos are L2 hits.
#include <atomic>

#include "c3c_internal.h"
#include "fuse_dev.h"

namespace c3c {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int BKC = 32;   // input channels per stage = K of one matrix-core step
constexpr int PIXB = 96;  // LDS bytes per staged pixel: 32 ch * 2 B + 32 B pad (bank-conflict-free B reads)

struct Args {
  const uint16_t* x;
  const uint16_t* cache;
  const u32x4* wpack;
  const uint16_t* bias;
  uint16_t* y;
  uint16_t* cache_out;
  int64_t hw;           // H * W
  int N, Ci, Co, T, Tc, H, W;
  int Kt, dt, p_l, Z, To, L;
  int chunks, cofrags;  // ceil(Ci / 32), ceil(Co / 16)
  uint32_t wpack_bytes;
  int tiles_co, tiles_w, tiles_h;
  int nblocks;
  int has_bias;
  int write_cache;
  // split-K: with splits > 1, workgroup split sp runs stages [sp nst / splits,
  // (sp + 1) nst / splits) of its tile and writes fp32 partial sums (no bias)
  // to part[sp][n][co][o][h][w]; splitk_reduce then adds them and the bias
  int splits;
  float* part;
  // the fused form (FU instances; NULL when absent): per-(n, ci) scale and
  // shift of the prologue, the residual added in the epilogue
  const float* scale;
  const float* shift;
  const uint16_t* residual;
};

// 8 channel rows of 8 pixels (v[c] = pixels 0..7 of channel c) -> 8 pixel
// records of 8 channels (o[p] = channels 0..7 of pixel p).
__device__ inline void transpose8x8(const u32x4 (&v)[8], u32x4 (&o)[8]) {
#pragma unroll
  for (int p = 0; p < 8; ++p) {
    const uint32_t sel = (p & 1) ? 0x07060302u : 0x05040100u;
#pragma unroll
    for (int r = 0; r < 4; ++r)
      o[p][r] = __builtin_amdgcn_perm(v[2 * r + 1][p >> 1], v[2 * r][p >> 1], sel);
  }
}

// Workgroup tile: BCO = 16*WCO*WAVES_CO output channels x BH = WR*WAVES_PX
// rows x BW = 16*WCF columns of one output frame.  Wave (wco, wpx) owns WCO
// x (WR*WCF) accumulator fragments of 16 x 16.  NBUF (2 or 3) LDS tile
// buffers: with 3, the barrier that publishes the next stage's tile sits
// inside the current stage, so the first operand reads of the next stage
// overlap the current stage's last matrix-core step.
// SPLIT: the split-K instance (a stage range per workgroup, fp32 partial
// sums out); a separate instance so that the unsplit kernel's register
// allocation is not shaped by the split epilogue.
// FU: the fused form.  0: none.  1: the residual only.  2: the prologue
// (and the residual when one is given).  With the prologue, each stage's
// scale / shift values load with its activations, and a stage whose frame
// comes from the new chunk gets the prologue on its staged registers, part
// by part as they arrive, before both the LDS store and the cache store see
// the values; positions outside the image keep their zero.  The residual
// joins the epilogue.
template <int WCO, int WR, int WCF, int WAVES_CO, int WAVES_PX, int NBUF, bool ALIGNED, bool SPLIT,
          int FU = 0>
__global__ __launch_bounds__(64 * WAVES_CO * WAVES_PX, 1) void conv3d_bf16(Args a) {
  constexpr int NT = 64 * WAVES_CO * WAVES_PX;
  constexpr bool PRO = FU == 2, RES = FU >= 1;
  constexpr int BH = WR * WAVES_PX, BW = 16 * WCF;
  constexpr int TH = BH + 2, TW = BW + 2;
  constexpr int NCH = BW / 8;                   // 8-pixel segments per tile row
  constexpr int NTASK = TH * NCH * (BKC / 8);   // (row, segment, 8-channel group)
  constexpr int TPT = (NTASK + NT - 1) / NT;
  constexpr int NHALO = TH * 2 * BKC;           // left / right halo column elements
  constexpr int HPT = (NHALO + NT - 1) / NT;
  constexpr int BUF = TH * TW * PIXB;
  constexpr int NPF = WR * WCF;                 // pixel fragments per wave
  static_assert(TW % 8 == 2, "the staging lane order assumes TW = 2 mod 8");
  static_assert(NBUF == 2 || NBUF == 3, "two or three tile buffers");
  // Lanes without a staging task or halo element still write, to a private
  // slot of a dummy region after the tile buffers: the tile write is then
  // free of branches, so it interleaves with the matrix-core steps and no
  // load is left outstanding on a skipped path.
  constexpr int DUMMY = NBUF * BUF;
  constexpr int DUMMY_BYTES = 64 * 16 + 7 * PIXB;
  static_assert(NBUF * BUF + DUMMY_BYTES <= 160 * 1024, "LDS tile buffers exceed 160 KiB");
  __shared__ __align__(16) unsigned char lds[NBUF * BUF + DUMMY_BYTES];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int wco = wave % WAVES_CO, wpx = wave / WAVES_CO;

  // ---- workgroup -> tile, XCD-contiguous
  int o, tw, th, n, ct, sp;
  {
    const int b = blockIdx.x;
    const int per = a.nblocks / 8, rem = a.nblocks % 8;
    const int xcd = b % 8, slot = b / 8;
    int L = (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + slot;
    o = L % a.To;
    L /= a.To;
    tw = L % a.tiles_w;
    L /= a.tiles_w;
    th = L % a.tiles_h;
    L /= a.tiles_h;
    n = L % a.N;
    L /= a.N;
    ct = SPLIT ? L % a.tiles_co : L;
    sp = SPLIT ? L / a.tiles_co : 0;
  }
  const int h0 = th * BH, w0 = tw * BW;

  // ---- active taps of this output frame (Eq. 4): source frame o + k dt - p_l in [0, Z)
  int k_lo = 0;
  while (k_lo < a.Kt && o + k_lo * a.dt - a.p_l < 0) ++k_lo;
  int k_hi = a.Kt - 1;
  while (k_hi >= 0 && o + k_hi * a.dt - a.p_l >= a.Z) --k_hi;
  // Stages run channel-chunk outer, tap inner: the workgroups of neighbouring
  // output frames (which share source frames) then read the same 32-channel
  // chunk of a frame close together in time, so the re-reads hit in L2.
  const int ntap = k_hi >= k_lo ? k_hi - k_lo + 1 : 0;
  const int nst = ntap * a.chunks;
  // this workgroup's share of the stages (all of them unless split-K)
  const int s_lo = SPLIT ? (sp * nst) / a.splits : 0;
  const int s_hi = SPLIT ? ((sp + 1) * nst) / a.splits : nst;
  const int cnt = s_hi - s_lo;
  constexpr uint32_t OOB = 0x80000000u;  // beyond every resource's size

  // One stage = (active tap k, 32-channel chunk c0).  Its activations are read
  // through a buffer resource that starts at channel c0 of source frame f and
  // ends after the last real channel, so every padding pixel and every
  // channel past Ci is an out-of-range offset and loads as 0; a chunk past
  // the last one has an empty resource.  wbase is the byte offset of the
  // stage's (kh, kw) = (0, 0) weight row in the packed weights.
  struct Stage {
    __amdgpu_buffer_rsrc_t rs;
    uint32_t cs;     // bytes between channel planes of the source
    uint32_t wbase;
    int k, c0, f;
  };
  auto stage_at = [&](int ki, int chunk) {
    Stage st;
    st.k = k_lo + ki;
    st.c0 = chunk * BKC;
    st.f = o + st.k * a.dt - a.p_l;
    // selects, not a branch: the stage loop stays one basic block
    const bool in_cache = st.f < a.Tc;
    const int64_t cstride = static_cast<int64_t>(in_cache ? a.Tc : a.T) * a.hw;
    const uint16_t* src = in_cache ? a.cache : a.x;
    const int64_t fr = in_cache ? st.f : st.f - a.Tc;
    const uint16_t* base = src + (static_cast<int64_t>(n) * a.Ci + st.c0) * cstride + fr * a.hw;
    int64_t bytes = ((a.Ci - 1 - st.c0) * cstride + a.hw) * 2;
    bytes = bytes > 0x7fffffff ? 0x7fffffff : bytes;
    bytes = bytes < 0 ? 0 : bytes;
    st.rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), 0,
                                              static_cast<int>(bytes), 0x00020000);
    st.cs = static_cast<uint32_t>(cstride * 2);
    st.wbase = static_cast<uint32_t>((st.k * 9 * a.chunks + chunk) * a.cofrags) * 1024u;
    return st;
  };

  // ---- per-thread staging constants.  A task is 8 channels (8g ..) x 8
  // pixels of one halo-tile row; tasks are numbered channel group fastest,
  // then row, so that the 8 lanes of one LDS write cycle (4 groups x 2 rows)
  // hit 8 distinct 16-byte bank groups.
  uint32_t t_g8[TPT], t_pix[TPT], t_lds[TPT];
  bool t_st[TPT], t_ok[TPT], t_in[TPT];
  int t_w[TPT];
#pragma unroll
  for (int tt = 0; tt < TPT; ++tt) {
    const int t = tid + tt * NT;
    const int g = t & 3, rr = (t >> 2) % TH, q = (t >> 2) / TH;
    const int gh = h0 - 1 + rr, w = w0 + 8 * q;
    t_st[tt] = (t < NTASK) & (rr < TH);
    // bitwise & (not &&): validity must become selects, not branches
    t_ok[tt] = t_st[tt] & (gh >= 0) & (gh < a.H) & (w < a.W);
    t_g8[tt] = static_cast<uint32_t>(8 * g);
    t_pix[tt] = static_cast<uint32_t>(gh * a.W + w) * 2u;
    t_lds[tt] = static_cast<uint32_t>((rr * TW + 1 + 8 * q) * PIXB + 16 * g);
    t_w[tt] = w;
    // interior rows of the tile (the cache write covers only those)
    t_in[tt] = t_st[tt] & (rr >= 1) & (rr <= BH) & (gh < a.H) & (w < a.W);
  }
  uint32_t h_ch[HPT], h_pix[HPT], h_lds[HPT];
  bool h_ok[HPT], h_in[HPT];
#pragma unroll
  for (int hh = 0; hh < HPT; ++hh) {
    const int e = tid + hh * NT;
    const int ch = e % BKC, side = (e / BKC) % 2, rr = e / (2 * BKC);
    const int gh = h0 - 1 + rr, gw = side ? w0 + BW : w0 - 1;
    h_in[hh] = e < NHALO;
    h_ok[hh] = h_in[hh] & (gh >= 0) & (gh < a.H) & (gw >= 0) & (gw < a.W);
    h_ch[hh] = static_cast<uint32_t>(ch);
    h_pix[hh] = static_cast<uint32_t>(gh * a.W + gw) * 2u;
    h_lds[hh] = static_cast<uint32_t>((rr * TW + (side ? TW - 1 : 0)) * PIXB + 2 * ch);
  }

  u32x4 sv[TPT][8];
  uint16_t hv[HPT];
  // PRO: this thread's 8 task channels (8g + j, the same g for every task
  // of a thread) and its halo channels, for the stage being loaded; batch
  // element n's scale / shift with channels past Ci out of range (0)
  float psc[8], psh[8], hsc[HPT], hsh[HPT];
  bool ppro = false;
  const __amdgpu_buffer_rsrc_t ssr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(PRO && a.scale ? a.scale + static_cast<int64_t>(n) * a.Ci : a.scale), 0,
      PRO && a.scale ? a.Ci * 4 : 0, 0x00020000);
  const __amdgpu_buffer_rsrc_t shr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(PRO && a.shift ? a.shift + static_cast<int64_t>(n) * a.Ci : a.shift), 0,
      PRO && a.shift ? a.Ci * 4 : 0, 0x00020000);

  // part p of a stage's loads: channel rows 2p, 2p + 1 of every task for
  // p = 0..3, the halo columns for p = 4 (spread over five steps so that no
  // burst of loads sits in front of the weight loads that follow it)
  auto load_stage = [&](const Stage& st, int part) {
    if (PRO && part == 0) {
      ppro = a.scale != nullptr && st.f >= a.Tc;
      const uint32_t c8 = static_cast<uint32_t>(st.c0) + t_g8[0];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        psc[j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(ssr, ppro ? (c8 + j) * 4u : OOB, 0, 0));
        psh[j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(shr, ppro ? (c8 + j) * 4u : OOB, 0, 0));
      }
#pragma unroll
      for (int hh = 0; hh < HPT; ++hh) {
        const uint32_t c = static_cast<uint32_t>(st.c0) + h_ch[hh];
        hsc[hh] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(ssr, ppro ? c * 4u : OOB, 0, 0));
        hsh[hh] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(shr, ppro ? c * 4u : OOB, 0, 0));
      }
    }
    if (part < 4)
#pragma unroll
    for (int tt = 0; tt < TPT; ++tt) {
      const uint32_t off = t_ok[tt] ? t_g8[tt] * st.cs + t_pix[tt] : OOB;
#pragma unroll
      for (int j = 2 * part; j < 2 * part + 2; ++j) {
        if (ALIGNED) {
          sv[tt][j] = __builtin_bit_cast(
              u32x4, __builtin_amdgcn_raw_buffer_load_b128(st.rs, off + j * st.cs, 0, 0));
        } else {
          uint32_t wd[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t o0 = (t_w[tt] + 2 * e < a.W) ? off + j * st.cs + 4u * e : OOB;
            const uint32_t o1 = (t_w[tt] + 2 * e + 1 < a.W) ? off + j * st.cs + 4u * e + 2u : OOB;
            const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(st.rs, o0, 0, 0);
            const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(st.rs, o1, 0, 0);
            wd[e] = (lo & 0xffffu) | (hi << 16);
          }
          sv[tt][j] = u32x4{wd[0], wd[1], wd[2], wd[3]};
        }
      }
    }
    if (part == 4)
#pragma unroll
    for (int hh = 0; hh < HPT; ++hh)
      hv[hh] = __builtin_amdgcn_raw_buffer_load_b16(
          st.rs, h_ok[hh] ? h_ch[hh] * st.cs + h_pix[hh] : OOB, 0, 0);
  };

  // PRO: the prologue on the staged registers of part `part` of a stage
  // (rows 2 part, 2 part + 1 of every task for part 0..3, the halo for part
  // 4), applied a few steps after that part's loads were issued so that the
  // VALU work interleaves with the matrix-core steps (branch-free: ppro is
  // false for a cache frame, and a task is in the image when t_ok; without
  // ALIGNED its pixels past W are padding too).
  auto pro_part = [&](int part) {
    if constexpr (PRO) {
      if (part < 4) {
#pragma unroll
        for (int tt = 0; tt < TPT; ++tt) {
          const bool ok = ppro & t_ok[tt];
#pragma unroll
          for (int j = 2 * part; j < 2 * part + 2; ++j) {
            if (ALIGNED) {
              sv[tt][j] = fuse_seg8(sv[tt][j], psc[j], psh[j], ok);
            } else {
#pragma unroll
              for (int r = 0; r < 4; ++r)
                sv[tt][j][r] = fuse_pair(sv[tt][j][r], psc[j], psh[j], ok & (t_w[tt] + 2 * r < a.W),
                                         ok & (t_w[tt] + 2 * r + 1 < a.W));
            }
          }
        }
      } else {
#pragma unroll
        for (int hh = 0; hh < HPT; ++hh) hv[hh] = fuse_one(hv[hh], hsc[hh], hsh[hh], ppro & h_ok[hh]);
      }
    }
  };

  // transpose the staged registers into LDS buffer `buf` (no branches:
  // lanes without a task or halo element write to their dummy slot)
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int tt = 0; tt < TPT; ++tt) {
      u32x4 pr[8];
      transpose8x8(sv[tt], pr);
      const uint32_t at = t_st[tt] ? static_cast<uint32_t>(buf * BUF) + t_lds[tt]
                                   : static_cast<uint32_t>(DUMMY + 16 * lane);
#pragma unroll
      for (int p = 0; p < 8; ++p)
        *reinterpret_cast<u32x4*>(lds + at + p * PIXB) = pr[p];
    }
#pragma unroll
    for (int hh = 0; hh < HPT; ++hh) {
      const uint32_t at = h_in[hh] ? static_cast<uint32_t>(buf * BUF) + h_lds[hh]
                                   : static_cast<uint32_t>(DUMMY + 2 * lane);
      *reinterpret_cast<uint16_t*>(lds + at) = hv[hh];
    }
  };

  // The designated workgroup writes its interior rows of a cache frame to
  // cache_out from the staging registers, through a buffer resource that ends
  // after the last real channel (stores at out-of-range offsets are dropped).
  // The condition is uniform over the workgroup.
  // The writers of a frame's chunks are spread over the output-channel tiles
  // (chunk c is written by tile c mod tiles_co), so that no tile carries the
  // whole cache write.
  auto cache_needed = [&](const Stage& st, bool real) {
    return a.write_cache && real && (st.c0 / BKC) % a.tiles_co == ct && st.f >= a.Z - a.L &&
           (st.k == a.Kt - 1 || o < a.dt);
  };
  auto cache_store = [&](const Stage& st) {
    const int64_t cstride = static_cast<int64_t>(a.L) * a.hw;
    uint16_t* cbase = a.cache_out + (static_cast<int64_t>(n) * a.Ci + st.c0) * cstride +
                      static_cast<int64_t>(st.f - (a.Z - a.L)) * a.hw;
    int64_t bytes = ((a.Ci - 1 - st.c0) * cstride + a.hw) * 2;
    bytes = bytes > 0x7fffffff ? 0x7fffffff : bytes;
    const __amdgpu_buffer_rsrc_t crs =
        __builtin_amdgcn_make_buffer_rsrc(cbase, 0, static_cast<int>(bytes), 0x00020000);
    const uint32_t ccs = static_cast<uint32_t>(cstride * 2);
#pragma unroll
    for (int tt = 0; tt < TPT; ++tt) {
      const uint32_t off = t_in[tt] ? t_g8[tt] * ccs + t_pix[tt] : OOB;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (ALIGNED) {
          __builtin_amdgcn_raw_buffer_store_b128(sv[tt][j], crs, off + j * ccs, 0, 0);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            __builtin_amdgcn_raw_buffer_store_b16(
                static_cast<uint16_t>(sv[tt][j][e >> 1] >> (16 * (e & 1))), crs,
                t_w[tt] + e < a.W ? off + j * ccs + 2u * e : OOB, 0, 0);
        }
      }
    }
  };

  // Weights of (kh, kw) step ij of a stage for this wave's fragments: one
  // 16-byte load per lane per fragment at wbase + ij * (bytes per (kh, kw)
  // row) + the fragment's offset.  Output-channel fragments past Co are
  // clamped to the last one: they only feed accumulator rows that are never
  // stored.  The prefetch for the stage after the last one reads row
  // (k_lo, chunk = chunks), which is still inside the packed weights.
  u32x4 wr[3][WCO];
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<u32x4*>(a.wpack), 0, static_cast<int>(a.wpack_bytes), 0x00020000);
  const uint32_t wrow = static_cast<uint32_t>(a.chunks * a.cofrags) * 1024u;
  const int cofrag0 = (ct * WAVES_CO + wco) * WCO;
  uint32_t wv[WCO];
#pragma unroll
  for (int cf = 0; cf < WCO; ++cf)
    wv[cf] = static_cast<uint32_t>(lane) * 16u +
             static_cast<uint32_t>(min(cofrag0 + cf, a.cofrags - 1)) * 1024u;
  // The bias of this lane's output channel in each fragment, all loaded
  // before the epilogue's first store: loaded fragment by fragment between
  // the stores, each load's wait also waited for every store before it.  The
  // plain aligned form loads them here and holds them through the main loop;
  // the fused and unaligned forms, whose main loops have no registers to
  // spare, at the start of the epilogue (with the residual batch).  A channel
  // past Co, or no bias: an out-of-range offset, 0.
  float bias_v[WCO] = {};
  auto load_bias = [&]() {
    const __amdgpu_buffer_rsrc_t brs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(a.bias), 0, a.has_bias ? a.Co * 2 : 0, 0x00020000);
#pragma unroll
    for (int cf = 0; cf < WCO; ++cf) {
      const uint32_t co = static_cast<uint32_t>((cofrag0 + cf) * 16 + (lane & 15));
      bias_v[cf] = __uint_as_float(static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b16(brs, 2u * co, 0, 0))
                                   << 16);
    }
  };
  if constexpr (!SPLIT && FU == 0 && ALIGNED) load_bias();
  auto load_w = [&](uint32_t wbase, int ij, u32x4 (&dst)[WCO]) {
    const uint32_t so = wbase + static_cast<uint32_t>(ij) * wrow;
#pragma unroll
    for (int cf = 0; cf < WCO; ++cf)
      dst[cf] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(wrs, wv[cf], so, 0));
  };

  f32x4 acc[WCO][NPF];
#pragma unroll
  for (int i = 0; i < WCO; ++i)
#pragma unroll
    for (int j = 0; j < NPF; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // per-lane LDS offset of this wave's activation operand (pixel l % 16,
  // channel group l / 16)
  const int lane_off = (wpx * WR * TW + (lane & 15)) * PIXB + (lane >> 4) * 16;

  // activation fragment pf of (kh, kw) step ij
  auto read_a = [&](const unsigned char* tile, int ij, int pf) {
    const int ki = ij / 3, kj = ij % 3, rp = pf / WCF, cfb = pf % WCF;
    return *reinterpret_cast<const u32x4*>(tile + ((rp + ki) * TW + cfb * 16 + kj) * PIXB);
  };

  u32x4 av[NPF];
  // (tap index, chunk) of the next stage, advanced incrementally
  int nk = SPLIT && ntap > 0 ? s_lo % ntap : 0, nc = SPLIT && ntap > 0 ? s_lo / ntap : 0;
  auto advance = [&]() {
    if (++nk == ntap) {
      nk = 0;
      ++nc;
    }
  };
  Stage cst = stage_at(nk, nc);
  if (cnt > 0) {
    load_w(cst.wbase, 0, wr[0]);
    load_w(cst.wbase, 1, wr[1]);
    for (int part = 0; part < 5; ++part) load_stage(cst, part);
    for (int part = 0; part < 5; ++part) pro_part(part);
    if (cache_needed(cst, true)) cache_store(cst);
    store_stage(0);
    __syncthreads();
#pragma unroll
    for (int pf = 0; pf < NPF; ++pf) av[pf] = read_a(lds + lane_off, 0, pf);
  }

  // Step (s, ij): the weights two steps ahead and part ij of the next
  // stage's activation loads are issued first; fragment pf's matrix-core
  // products are followed by the re-read of that fragment for the next step
  // (or, with three buffers, for step 0 of the next stage, whose tile was
  // published by the barrier at the end of step 7).  Loads for a stage past
  // the last one are issued anyway and read zeros (an empty resource):
  // keeping them unconditional keeps the step one basic block that the
  // explicit interleave can schedule.
  int cur = 0;
  for (int s = 0; s < cnt; ++s) {
    advance();
    const Stage nst_ = stage_at(nk, nc);
    const int nxt = cur + 1 == NBUF ? 0 : cur + 1;
    const unsigned char* tile = lds + cur * BUF + lane_off;
    const unsigned char* ntile = lds + nxt * BUF + lane_off;
#pragma unroll
    for (int ij = 0; ij < 9; ++ij) {
      // the cache write (rare, workgroup-uniform) is its own block ahead of
      // the scheduled region of step 7
      // PRO: the next stage's prologue, part p at step p + 3 (its loads were
      // issued at step p), the halo at step 6; all before the cache and LDS
      // stores of step 7
      if (PRO && ij >= 3 && ij <= 6) pro_part(ij - 3);
      if (PRO && ij == 6) pro_part(4);
      if (ij == 7 && cache_needed(nst_, s + 1 < cnt)) cache_store(nst_);
      // keep every LDS read inside its own step: re-reading is cheaper in
      // registers than keeping overlapping rows of neighbouring kh live
      asm volatile("" ::: "memory");
      __builtin_amdgcn_sched_barrier(0);
      load_w(ij + 2 < 9 ? cst.wbase : nst_.wbase, (ij + 2) % 9, wr[(ij + 2) % 3]);
      if (ij < 5) load_stage(nst_, ij);
      // The buffer written here was last read two stages ago (three
      // buffers) or in the previous stage (two buffers); a barrier has
      // passed since in both cases.
      if (ij == 7) store_stage(nxt);
#pragma unroll
      for (int pf = 0; pf < NPF; ++pf) {
#pragma unroll
        for (int cf = 0; cf < WCO; ++cf)
          acc[cf][pf] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(bf16x8, av[pf]), __builtin_bit_cast(bf16x8, wr[ij % 3][cf]),
              acc[cf][pf], 0, 0, 0);
        if (ij + 1 < 9)
          av[pf] = read_a(tile, ij + 1, pf);
        else if (NBUF == 3)
          av[pf] = read_a(ntile, 0, pf);
      }
      // explicit interleave (masks: 0x008 MFMA, 0x100 DS read, 0x020 VMEM
      // read, 0x200 DS write): after each fragment's products, its re-read;
      // global reads spread over the first groups, LDS writes over all
      constexpr int nvm_stage = 2 * TPT;
      const int nvm = WCO + (ij < 4 ? nvm_stage : ij == 4 ? HPT : 0);
      const int ndw = ij == 7 ? TPT * 8 + HPT : 0;
      const bool rd = ij + 1 < 9 || NBUF == 3;
      for (int g = 0; g < NPF; ++g) {
        __builtin_amdgcn_sched_group_barrier(0x008, WCO, 0);
        if (rd) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        for (int q = (nvm * g) / NPF; q < (nvm * (g + 1)) / NPF; ++q)
          __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        for (int q = (ndw * g) / NPF; q < (ndw * (g + 1)) / NPF; ++q)
          __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
      }
      if (NBUF == 3 && ij == 7) __syncthreads();
    }
    if (NBUF == 2) {
      __syncthreads();
#pragma unroll
      for (int pf = 0; pf < NPF; ++pf) av[pf] = read_a(ntile, 0, pf);
    }
    cst = nst_;
    cur = nxt;
  }

  // ---- epilogue: bias once, round to bf16, NCTHW store.  With the
  // activations as the A operand, lane l holds output channel l % 16 for the
  // four consecutive pixels 4 * (l / 16) .. + 3 of each fragment: one 8-byte
  // store per fragment.  Under split-K the fp32 sums go to the partial
  // buffer instead (one 16-byte store per fragment), without the bias.
  const int64_t plane = static_cast<int64_t>(a.To) * a.hw;
  if constexpr (SPLIT) {
    float* pbase = a.part + (static_cast<int64_t>(sp) * a.N + n) * a.Co * plane +
                   static_cast<int64_t>(o) * a.hw;
#pragma unroll
    for (int cf = 0; cf < WCO; ++cf) {
      const int co = (cofrag0 + cf) * 16 + (lane & 15);
#pragma unroll
      for (int pf = 0; pf < NPF; ++pf) {
        const int h = h0 + wpx * WR + pf / WCF, w = w0 + (pf % WCF) * 16 + 4 * (lane >> 4);
        if (co >= a.Co || h >= a.H || w >= a.W) continue;
        float* dst = pbase + co * plane + static_cast<int64_t>(h) * a.W + w;
        if (ALIGNED && w + 4 <= a.W) {
          *reinterpret_cast<f32x4*>(dst) = acc[cf][pf];
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (w + r < a.W) dst[r] = acc[cf][pf][r];
        }
      }
    }
    return;
  }
  uint16_t* ybase = a.y + (static_cast<int64_t>(n) * a.Co) * plane + static_cast<int64_t>(o) * a.hw;
  // RES: every fragment's residual values, loaded as one batch before any
  // store (branch-free: a position outside the output reads the residual's
  // first element and is not used), so the block waits for memory once
  if constexpr (FU != 0 || !ALIGNED) load_bias();
  uint2 rv[RES ? WCO : 1][RES ? NPF : 1];
  if constexpr (RES) {
    const bool has_r = a.residual != nullptr;
#pragma unroll
    for (int cf = 0; cf < WCO; ++cf) {
      const int co = (cofrag0 + cf) * 16 + (lane & 15);
#pragma unroll
      for (int pf = 0; pf < NPF; ++pf) {
        const int h = h0 + wpx * WR + pf / WCF, w = w0 + (pf % WCF) * 16 + 4 * (lane >> 4);
        const bool ok = has_r & (co < a.Co) & (h < a.H) & (w < a.W);
        const int64_t off = (static_cast<int64_t>(n) * a.Co + (ok ? co : 0)) * plane +
                            static_cast<int64_t>(o) * a.hw + (ok ? static_cast<int64_t>(h) * a.W + w : 0);
        const uint16_t* rsrc = has_r ? a.residual + off : a.y;
        if (ALIGNED) {
          rv[cf][pf] = *reinterpret_cast<const uint2*>(rsrc);
        } else {
          uint16_t e[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) e[r] = rsrc[ok & (w + r < a.W) ? r : 0];
          rv[cf][pf] = make_uint2(e[0] | (static_cast<uint32_t>(e[1]) << 16), e[2] | (static_cast<uint32_t>(e[3]) << 16));
        }
      }
    }
  }
#pragma unroll
  for (int cf = 0; cf < WCO; ++cf) {
    const int co = (cofrag0 + cf) * 16 + (lane & 15);
    const float bb = bias_v[cf];
#pragma unroll
    for (int pf = 0; pf < NPF; ++pf) {
      const int h = h0 + wpx * WR + pf / WCF, w = w0 + (pf % WCF) * 16 + 4 * (lane >> 4);
      if (co >= a.Co || h >= a.H || w >= a.W) continue;
      uint16_t* dst = ybase + co * plane + static_cast<int64_t>(h) * a.W + w;
      // RES: the residual at the same position, added before the rounding
      f32x4 rr = {0.f, 0.f, 0.f, 0.f};
      if (RES && a.residual) {
        const uint2 r2 = rv[RES ? cf : 0][RES ? pf : 0];
        rr = f32x4{fuse_widen(r2.x & 0xffffu), fuse_widen(r2.x >> 16), fuse_widen(r2.y & 0xffffu),
                   fuse_widen(r2.y >> 16)};
      }
      // one round-to-nearest-even conversion per value (hardware, two at a time)
      const uint32_t v01 = __builtin_bit_cast(
          uint32_t, __builtin_convertvector((f32x2{acc[cf][pf][0] + bb + rr[0], acc[cf][pf][1] + bb + rr[1]}), bf16x2));
      const uint32_t v23 = __builtin_bit_cast(
          uint32_t, __builtin_convertvector((f32x2{acc[cf][pf][2] + bb + rr[2], acc[cf][pf][3] + bb + rr[3]}), bf16x2));
      if (ALIGNED && w + 4 <= a.W) {
        *reinterpret_cast<uint2*>(dst) = make_uint2(v01, v23);
      } else {
        const uint16_t v[4] = {static_cast<uint16_t>(v01), static_cast<uint16_t>(v01 >> 16),
                               static_cast<uint16_t>(v23), static_cast<uint16_t>(v23 >> 16)};
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (w + r < a.W) dst[r] = v[r];
      }
    }
  }
}

// Split-K reduction: y = bf16(sum of the splits' partial sums + bias), each
// element summed in split order (deterministic), the bias added once, one
// round-to-nearest-even.  Four consecutive elements of one output-channel
// plane per thread when the plane length is a multiple of 4.
template <bool VEC4>
__global__ __launch_bounds__(256) void splitk_reduce(const float* __restrict__ part,
                                                     const uint16_t* __restrict__ bias,
                                                     const uint16_t* residual,
                                                     uint16_t* y, int64_t total,
                                                     int64_t plane, int Co, int splits,
                                                     int has_bias) {
  constexpr int V = VEC4 ? 4 : 1;
  for (int64_t i = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * V; i < total;
       i += static_cast<int64_t>(gridDim.x) * 256 * V) {
    const int co = static_cast<int>((i / plane) % Co);
    const float bb = has_bias ? __uint_as_float(static_cast<uint32_t>(bias[co]) << 16) : 0.f;
    if constexpr (VEC4) {
      f32x4 v = *reinterpret_cast<const f32x4*>(part + i);
      for (int s = 1; s < splits; ++s)
        v += *reinterpret_cast<const f32x4*>(part + static_cast<int64_t>(s) * total + i);
      if (residual) {  // the fused form's residual, after the split sums (y may be the residual)
        const uint2 r2 = *reinterpret_cast<const uint2*>(residual + i);
        v += f32x4{fuse_widen(r2.x & 0xffffu), fuse_widen(r2.x >> 16), fuse_widen(r2.y & 0xffffu),
                   fuse_widen(r2.y >> 16)};
      }
      const uint32_t v01 = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{v[0] + bb, v[1] + bb}), bf16x2));
      const uint32_t v23 = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{v[2] + bb, v[3] + bb}), bf16x2));
      *reinterpret_cast<uint2*>(y + i) = make_uint2(v01, v23);
    } else {
      float v = part[i];
      for (int s = 1; s < splits; ++s) v += part[static_cast<int64_t>(s) * total + i];
      if (residual) v += fuse_widen(residual[i]);
      const uint32_t r = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{v + bb, 0.f}), bf16x2));
      y[i] = static_cast<uint16_t>(r);
    }
  }
}

// Tile configurations of the bf16 kernel (template arguments of run()).
enum Cfg { CFG_C192, CFG_C96, CFG_C16, CFG_C160_4X80, CFG_C160_10X32, CFG_C128_4X80, CFG_C64_4X64 };

// Launch plan of one bf16 fast call: tile configuration, workgroups of one
// split, split-K factor, and the fp32 partial-sum bytes the split needs.
struct Plan {
  Cfg cfg;
  int64_t tiles_co, tiles_w, tiles_h, blocks;
  int64_t tile_flop_px;  // output channels x pixels of one tile
  int splits;
  int64_t part_bytes;
};

void set_tiles(const Geo& g, int64_t bco, int64_t bh, int64_t bw, Plan* p) {
  p->tiles_co = (g.d.Co + bco - 1) / bco;
  p->tiles_w = (g.Wo + bw - 1) / bw;
  p->tiles_h = (g.Ho + bh - 1) / bh;
  p->blocks = p->tiles_co * p->tiles_w * p->tiles_h * g.To * g.d.N;
  p->tile_flop_px = bco * bh * bw;
}

template <int WCO, int WR, int WCF, int WAVES_CO, int WAVES_PX, int NBUF>
hipError_t run(const Geo& g, Args a, const Plan& p, bool aligned, int fused, hipStream_t s,
               LaunchInfo* info) {
  a.tiles_co = static_cast<int>(p.tiles_co);
  a.tiles_w = static_cast<int>(p.tiles_w);
  a.tiles_h = static_cast<int>(p.tiles_h);
  const int64_t blocks = p.blocks * a.splits;
  if (info) {
    info->kernel = C3C_KERNEL_CONV3D_BF16;
    info->tile_co = 16 * WCO * WAVES_CO;
    info->tile_h = WR * WAVES_PX;
    info->tile_w = 16 * WCF;
    info->workgroups = blocks;
    info->splits = a.splits;
    info->cache_in_kernel = a.write_cache != 0;
    return hipSuccess;
  }
  if (blocks == 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  a.nblocks = static_cast<int>(blocks);
  const dim3 grid(static_cast<unsigned>(blocks)), block(64 * WAVES_CO * WAVES_PX);
  const bool split = a.splits > 1;
#define C3C_BF16(AL, SP, FU)                                                                        \
  if (aligned == AL && split == SP && fused == FU)                                                   \
    hipLaunchKernelGGL((conv3d_bf16<WCO, WR, WCF, WAVES_CO, WAVES_PX, NBUF, AL, SP, FU>), grid, block, 0, s, a);
  C3C_BF16(true, false, 0) C3C_BF16(false, false, 0) C3C_BF16(true, true, 0) C3C_BF16(false, true, 0)
  C3C_BF16(true, false, 1) C3C_BF16(false, false, 1) C3C_BF16(true, true, 1) C3C_BF16(false, true, 1)
  C3C_BF16(true, false, 2) C3C_BF16(false, false, 2) C3C_BF16(true, true, 2) C3C_BF16(false, true, 2)
#undef C3C_BF16
  if (!split) return hipGetLastError();
  const int64_t plane = static_cast<int64_t>(a.To) * a.hw;
  const int64_t total = static_cast<int64_t>(a.N) * a.Co * plane;
  const bool vec4 = plane % 4 == 0 && (reinterpret_cast<uintptr_t>(a.y) & 7u) == 0;
  int64_t rb = (total / (vec4 ? 4 : 1) + 255) / 256;
  if (rb > 65536) rb = 65536;
  const uint16_t* res = fused != 0 ? a.residual : nullptr;
  if (vec4 && (res == nullptr || (reinterpret_cast<uintptr_t>(res) & 7u) == 0))
    hipLaunchKernelGGL(splitk_reduce<true>, dim3(static_cast<unsigned>(rb)), dim3(256), 0, s, a.part,
                       a.bias, res, a.y, total, plane, a.Co, a.splits, a.has_bias);
  else
    hipLaunchKernelGGL(splitk_reduce<false>, dim3(static_cast<unsigned>(rb)), dim3(256), 0, s, a.part,
                       a.bias, res, a.y, total, plane, a.Co, a.splits, a.has_bias);
  return hipGetLastError();
}

// Every frame of the new cache must be the source of some (output frame,
// tap) pair for the fused cache write to cover it.
bool cache_covered(const Geo& g) {
  for (int64_t f = g.Z - g.L; f < g.Z; ++f) {
    bool hit = false;
    for (int64_t k = 0; k < g.d.Kt && !hit; ++k) {
      const int64_t o = f + g.p_l - k * g.d.dil_t;
      hit = o >= 0 && o < g.To;
    }
    if (!hit) return false;
  }
  return true;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

// compute units of the current device (queried once per device)
int64_t device_compute_units() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cache[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cache[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

namespace {

int64_t compute_units() { return device_compute_units(); }

// The tile configuration by output-channel count, and the split-K factor: a
// call whose workgroups fill less than one round of the compute units splits
// each tile's stages over S workgroups when the modelled time (microseconds)
//   rounds(blocks * S) * (stages per split + 3) * t_stage
//   + (S > 1) * (2 * S * output elements * 4 B / 5 TB/s + 5)
// is lower than unsplit.  t_stage is one stage's FLOP (2 * 288 * tile) at
// 6.9 TFLOP/s per compute unit, the measured main-loop rate; 3 stages stand
// for a workgroup's fixed cost; the last term is the fp32 partial sums
// written and read back, and the reduction launch.
Plan plan_bf16(const Geo& g) {
  Plan p;
  const int64_t Co = g.d.Co;
  const int64_t cus = compute_units();
  if (Co > 128 && Co % 192 == 0) {
    p.cfg = CFG_C192;
    set_tiles(g, 192, 4, 64, &p);
  } else if (Co <= 16) {
    // a head conv with a few output channels (e.g. 3, to RGB): one 16-channel
    // fragment per wave on an 8 x 64 tile, 1/6 of the matrix-core work of a
    // 96-channel tile
    p.cfg = CFG_C16;
    set_tiles(g, 16, 8, 64, &p);
  } else if (Co <= 96) {
    // 96 channels x 6 x 64 pixels on 2 x 2 waves (48 channels x 3 rows each):
    // each weight fragment is fetched by two waves, not four, and the smaller
    // halo tile leaves room for three LDS buffers
    p.cfg = CFG_C96;
    set_tiles(g, 96, 6, 64, &p);
  } else {
    // 160-channel tiles of 4 x 80 or 10 x 32 pixels.  A workgroup of either
    // shape takes about the same time (measured), so the shape with fewer
    // rounds of workgroups over the device's compute units wins; on a tie,
    // 4 x 80 (half the halo-column loads).
    Plan q;
    set_tiles(g, 160, 4, 80, &p);
    set_tiles(g, 160, 10, 32, &q);
    if ((p.blocks + cus - 1) / cus <= (q.blocks + cus - 1) / cus) {
      p.cfg = CFG_C160_4X80;
    } else {
      p = q;
      p.cfg = CFG_C160_10X32;
    }
    // 128-channel 4 x 80 tiles when they pad the output channels no more
    // than the 160-channel tiles do and take less time in whole rounds of
    // workgroups (rounds x channels per tile; a 128-channel workgroup does
    // 4/5 of a 160-channel one's work): a layer whose 160-channel tiles
    // leave part of the device idle in its last round (640 -> 640 at 44 x 80:
    // 176 workgroups on 256 compute units; 220 with 128 channels, same round)
    Plan r;
    set_tiles(g, 128, 4, 80, &r);
    if (r.tiles_co * 128 <= p.tiles_co * 160 &&
        ((r.blocks + cus - 1) / cus) * 128 < ((p.blocks + cus - 1) / cus) * 160) {
      p = r;
      p.cfg = CFG_C128_4X80;
    }
  }
  p.splits = 1;
  p.part_bytes = 0;
  if (p.blocks > 0 && p.blocks < cus) {
    int64_t ntap = 0;  // most active taps of any output frame (Eq. 4)
    for (int64_t o = 0; o < g.To; ++o) {
      int64_t n = 0;
      for (int64_t k = 0; k < g.d.Kt; ++k) {
        const int64_t f = o + k * g.d.dil_t - g.p_l;
        n += f >= 0 && f < g.Z;
      }
      ntap = n > ntap ? n : ntap;
    }
    const int64_t nst = ntap * ((g.d.Ci + BKC - 1) / BKC);
    const double t_stage = 2.0 * 9 * BKC * static_cast<double>(p.tile_flop_px) / 6.9e6;
    const double out_elems = static_cast<double>(g.d.N * Co * g.To * g.Ho * g.Wo);
    auto cost = [&](int64_t S) {
      const double rounds = static_cast<double>((p.blocks * S + cus - 1) / cus);
      return rounds * static_cast<double>((nst + S - 1) / S + 3) * t_stage +
             (S > 1 ? 2.0 * static_cast<double>(S) * out_elems * 4.0 / 5e6 + 5.0 : 0.0);
    };
    int64_t best = 1;
    for (int64_t S = 2; S <= 8; ++S)
      if (nst / S >= 4 && cost(S) < cost(best)) best = S;
    p.splits = static_cast<int>(best);
    if (best > 1) p.part_bytes = best * g.d.N * Co * g.To * g.Ho * g.Wo * 4;
  }
  return p;
}

// The plan of a call that runs unsplit (no workspace, or too small a one)
// whose tiles fill less than one round of the compute units: of its own
// tiling, the 128-channel 4 x 80 tiling (from the 192-channel one, when it
// pads no more output channels) and the 64-channel 4 x 64 tiling, the one of
// least modelled time
//   rounds of workgroups x the tile's output channels x pixels x c,
// c = 1 for the 192-, 160- and 128-channel tiles and 1.7 for the 64-channel
// tile: with two output-channel fragments per wave, each activation operand
// read from LDS feeds two products instead of four to six, and its main loop
// runs at about 4.0 TFLOP/s per compute unit against 6.9.  Measured, one
// output frame from two cached ones: 384 -> 384 at 60 x 104, 0.133 ms on 90
// workgroups of 128 x 4x80, 0.092 on 180 of 64 x 4x64; 192 -> 192 at 60 x
// 104, 0.087 on 30 of 192 x 4x64, 0.048 on 90 of 64 x 4x64.  With two output
// frames the first stays on 128 x 4x80 (180 workgroups, 0.139 ms, against two
// rounds of 360, 0.162).  Every output element's products are accumulated in
// the same order on every tile, so the outputs are bit-identical.  A call
// that splits keeps the tiling its split-K model is set for, and
// C3C_MODE_CHANNEL_TILES keeps the output-channel tiling.
Plan unsplit_plan(const Geo& g, Plan p) {
  const int64_t cus = compute_units();
  p.splits = 1;
  p.part_bytes = 0;
  const bool wide = p.cfg == CFG_C192 || p.cfg == CFG_C160_4X80 || p.cfg == CFG_C160_10X32 ||
                    p.cfg == CFG_C128_4X80;
  if (g.channel_tiles || !wide || p.blocks >= cus) return p;
  // cost in tenths of c
  auto cost = [&](const Plan& q, int64_t c10) {
    return (q.blocks + cus - 1) / cus * q.tile_flop_px * c10;
  };
  int64_t best = cost(p, 10);
  if (p.cfg == CFG_C192) {
    Plan r;
    set_tiles(g, 128, 4, 80, &r);
    if (r.tiles_co * 128 <= p.tiles_co * 192 && cost(r, 10) < best) {
      r.cfg = CFG_C128_4X80;
      r.splits = 1;
      r.part_bytes = 0;
      p = r;
      best = cost(r, 10);
    }
  }
  Plan q;
  set_tiles(g, 64, 4, 64, &q);
  if (cost(q, 17) < best) {
    q.cfg = CFG_C64_4X64;
    q.splits = 1;
    q.part_bytes = 0;
    p = q;
  }
  return p;
}

}  // namespace

int64_t fast_bf16_workspace_bytes(const Geo& g) { return plan_bf16(g).part_bytes; }

hipError_t launch_fast_bf16(const Geo& g, const void* x, const void* cache, const void* wpack,
                            const void* bias, void* y, void* cache_out, void* ws,
                            int64_t ws_bytes, bool* cache_written, hipStream_t s, const Fuse& fu,
                            LaunchInfo* info) {
  const PackDims p = pack_dims(g.d);
  Args a;
  a.x = static_cast<const uint16_t*>(x);
  a.cache = static_cast<const uint16_t*>(cache);
  a.wpack = static_cast<const u32x4*>(wpack);
  a.bias = static_cast<const uint16_t*>(bias);
  a.y = static_cast<uint16_t*>(y);
  a.cache_out = static_cast<uint16_t*>(cache_out);
  a.hw = g.d.H * g.d.W;
  a.N = static_cast<int>(g.d.N);
  a.Ci = static_cast<int>(g.d.Ci);
  a.Co = static_cast<int>(g.d.Co);
  a.T = static_cast<int>(g.d.T);
  a.Tc = static_cast<int>(g.d.Tc);
  a.H = static_cast<int>(g.d.H);
  a.W = static_cast<int>(g.d.W);
  a.Kt = static_cast<int>(g.d.Kt);
  a.dt = static_cast<int>(g.d.dil_t);
  a.p_l = static_cast<int>(g.p_l);
  a.Z = static_cast<int>(g.Z);
  a.To = static_cast<int>(g.To);
  a.L = static_cast<int>(g.L);
  a.chunks = static_cast<int>(p.chunks);
  a.cofrags = static_cast<int>(p.cofrags);
  a.wpack_bytes = static_cast<uint32_t>(p.elems() * 2);
  // 32-bit buffer offsets: one 32-channel chunk of a source or cache frame
  // and the packed weights must each span less than 2 GiB
  int64_t frames = g.d.T > g.d.Tc ? g.d.T : g.d.Tc;
  if (g.L > frames) frames = g.L;
  if (static_cast<int64_t>(BKC) * frames * a.hw * 2 >= 0x7fffffff || p.elems() * 2 >= 0x7fffffff)
    return hipErrorInvalidValue;
  a.has_bias = g.d.has_bias ? 1 : 0;
  a.write_cache = (g.L > 0 && cache_covered(g)) ? 1 : 0;
  *cache_written = a.write_cache != 0;
  a.scale = fu.scale;
  a.shift = fu.shift;
  a.residual = fu.residual;
  // instance: 0 plain, 1 residual only, 2 prologue (+ residual)
  const int fused = fu.pro() ? 2 : fu.residual ? 1 : 0;
  const bool aligned = (g.d.W % 8 == 0) && (x == nullptr || aligned16(x)) &&
                       (cache == nullptr || aligned16(cache)) &&
                       (cache_out == nullptr || aligned16(cache_out)) &&
                       (fu.residual == nullptr || (reinterpret_cast<uintptr_t>(fu.residual) & 7u) == 0);
  Plan pl = plan_bf16(g);
  // split-K only with a large enough, 16-byte-aligned workspace; else unsplit
  const bool split = pl.splits > 1 && ws != nullptr && ws_bytes >= pl.part_bytes &&
                     (reinterpret_cast<uintptr_t>(ws) & 15u) == 0;
  if (!split) pl = unsplit_plan(g, pl);
  a.splits = split ? pl.splits : 1;
  a.part = split ? static_cast<float*>(ws) : nullptr;
  switch (pl.cfg) {
    case CFG_C192: return run<6, 2, 4, 2, 2, 3>(g, a, pl, aligned, fused, s, info);
    case CFG_C96: return run<3, 3, 4, 2, 2, 3>(g, a, pl, aligned, fused, s, info);
    case CFG_C16: return run<1, 2, 4, 1, 4, 2>(g, a, pl, aligned, fused, s, info);
    // two LDS buffers measured 1.4-3.4% faster than three on the 720p
    // layers for this tile (the 192- and 96-channel tiles keep three)
    case CFG_C160_4X80: return run<5, 2, 5, 2, 2, 2>(g, a, pl, aligned, fused, s, info);
    case CFG_C128_4X80: return run<4, 2, 5, 2, 2, 2>(g, a, pl, aligned, fused, s, info);
    // two fragments per wave: 64 x 4x64 tiles for unsplit calls that fill few compute units
    case CFG_C64_4X64: return run<2, 2, 4, 2, 2, 3>(g, a, pl, aligned, fused, s, info);
    default: return run<5, 5, 2, 2, 2, 3>(g, a, pl, aligned, fused, s, info);
  }
}

}  // namespace c3c
