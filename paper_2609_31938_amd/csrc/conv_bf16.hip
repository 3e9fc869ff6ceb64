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
//   * Weights (A) come pre-packed in fragment order (c3c_weight_repack): one
//     16-byte load per lane per fragment, straight from L2 into registers,
//     two kernel taps ahead of their use (a 3-slot register ring).
//   * Activations (B) are staged per (tap, 32-channel chunk) as a halo tile
//     [BH+2][BW+2][32 ch] in LDS, channel-innermost with an 80-byte pixel
//     pitch, so that each lane reads its 8 K-consecutive channels with one
//     ds_read_b128 and the nine (kh, kw) offsets of the 3x3 kernel are nine
//     immediate address offsets into the same tile.  Global reads are
//     16-byte row segments of the NCTHW planes; an 8x8 register transpose
//     (v_perm) turns 8 channel rows x 8 pixels into 8 pixel records.  The
//     tile is double-buffered: the next stage's global loads are in flight
//     while the current stage computes.
//   * Workgroups are numbered so that each of the 8 XCDs (which take
//     workgroups round-robin) runs a contiguous range of tiles -- consecutive
//     output frames of the same spatial tile, then neighbouring tiles -- so
//     the frames shared by neighbouring taps and the halos are L2 hits.
#include "c3c_internal.h"

namespace c3c {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

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
};

__device__ inline uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

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
// x (WR*WCF) accumulator fragments of 16 x 16.
template <int WCO, int WR, int WCF, int WAVES_CO, int WAVES_PX, bool ALIGNED>
__global__ __launch_bounds__(64 * WAVES_CO * WAVES_PX, 1) void conv3d_bf16(Args a) {
  constexpr int NT = 64 * WAVES_CO * WAVES_PX;
  constexpr int BH = WR * WAVES_PX, BW = 16 * WCF;
  constexpr int TH = BH + 2, TW = BW + 2;
  constexpr int TH4 = (TH + 3) / 4 * 4;
  constexpr int NCH = BW / 8;                   // 8-pixel segments per tile row
  constexpr int NTASK = TH4 * NCH * (BKC / 8);  // (row, segment, 8-channel group)
  constexpr int TPT = (NTASK + NT - 1) / NT;
  constexpr int NHALO = TH * 2 * BKC;           // left / right halo column elements
  constexpr int HPT = (NHALO + NT - 1) / NT;
  constexpr int BUF = TH * TW * PIXB;
  constexpr int NPF = WR * WCF;                 // pixel fragments per wave
  static_assert(TW % 8 == 2, "the staging lane order assumes TW = 2 mod 8");
  __shared__ __align__(16) unsigned char lds[2 * BUF];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int wco = wave % WAVES_CO, wpx = wave / WAVES_CO;

  // ---- workgroup -> tile, XCD-contiguous
  int o, tw, th, n, ct;
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
    ct = L / a.N;
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

  const int cofrag0 = (ct * WAVES_CO + wco) * WCO;

  // ---- staging task decode: lane bits (g0, r0, r1, g1) first so that the
  // 8 lanes of one LDS write cycle hit 8 distinct 16-byte bank groups
  auto task = [&](int t, int& g, int& rr, int& q) {
    g = (t & 1) | (((t >> 3) & 1) << 1);
    rr = ((t >> 1) & 3) | (((t >> 4) % (TH4 / 4)) << 2);
    q = (t >> 4) / (TH4 / 4);
  };

  u32x4 sv[TPT][8];
  uint16_t hv[HPT];

  // Stage s reads the 32-channel chunk c0 of source frame f through a buffer
  // resource that ends after the last real channel, so that every padding
  // pixel and every channel past Ci is an out-of-range offset and loads as 0.
  auto stage_src = [&](int s, int& f, int& c0, int& k, __amdgpu_buffer_rsrc_t& rs,
                       uint32_t& cs_bytes) {
    k = k_lo + s % ntap;
    c0 = (s / ntap) * BKC;
    f = o + k * a.dt - a.p_l;
    const uint16_t* base;
    int64_t cstride;
    if (f < a.Tc) {
      cstride = static_cast<int64_t>(a.Tc) * a.hw;
      base = a.cache + (static_cast<int64_t>(n) * a.Ci + c0) * cstride + f * a.hw;
    } else {
      cstride = static_cast<int64_t>(a.T) * a.hw;
      base = a.x + (static_cast<int64_t>(n) * a.Ci + c0) * cstride + (f - a.Tc) * a.hw;
    }
    int64_t bytes = ((a.Ci - 1 - c0) * cstride + a.hw) * 2;
    if (bytes > 0x7fffffff) bytes = 0x7fffffff;
    if (bytes < 0) bytes = 0;  // a stage past the last one: every load reads 0
    rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), 0,
                                           static_cast<int>(bytes), 0x00020000);
    cs_bytes = static_cast<uint32_t>(cstride * 2);
  };
  constexpr uint32_t OOB = 0x80000000u;  // beyond every resource's size

  // part p of stage s's loads: channel rows 2p, 2p + 1 of every task for
  // p = 0..3, the halo columns for p = 4 (spread over five steps so that no
  // burst of loads sits in front of the weight loads that follow it)
  auto load_stage = [&](int s, int part) {
    int f, c0, k;
    __amdgpu_buffer_rsrc_t rs;
    uint32_t cs;
    stage_src(s, f, c0, k, rs, cs);
    if (part < 4)
#pragma unroll
    for (int tt = 0; tt < TPT; ++tt) {
      const int t = tid + tt * NT;
      int g, rr, q;
      task(t, g, rr, q);
      const int gh = h0 - 1 + rr, w = w0 + 8 * q;
      // bitwise & (not &&): validity must become selects, not branches
      const bool rowok = (t < NTASK) & (rr < TH) & (gh >= 0) & (gh < a.H);
      const uint32_t off = static_cast<uint32_t>(8 * g) * cs +
                           static_cast<uint32_t>(gh * a.W + w) * 2u;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (j / 2 != part) continue;
        const bool chok = rowok & (c0 + 8 * g + j < a.Ci);
        if (ALIGNED) {
          const uint32_t oj = (chok & (w < a.W)) ? off + j * cs : OOB;
          sv[tt][j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, oj, 0, 0));
        } else {
          uint32_t wd[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t o0 = (chok & (w + 2 * e < a.W)) ? off + j * cs + 4u * e : OOB;
            const uint32_t o1 = (chok & (w + 2 * e + 1 < a.W)) ? off + j * cs + 4u * e + 2u : OOB;
            const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(rs, o0, 0, 0);
            const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(rs, o1, 0, 0);
            wd[e] = (lo & 0xffffu) | (hi << 16);
          }
          sv[tt][j] = u32x4{wd[0], wd[1], wd[2], wd[3]};
        }
      }
    }
    if (part == 4)
#pragma unroll
    for (int hh = 0; hh < HPT; ++hh) {
      const int e = tid + hh * NT;
      const int ch = e % BKC, side = (e / BKC) % 2, rr = e / (2 * BKC);
      const int gh = h0 - 1 + rr, gw = side ? w0 + BW : w0 - 1;
      const bool ok = (e < NHALO) & (gh >= 0) & (gh < a.H) & (gw >= 0) & (gw < a.W) & (c0 + ch < a.Ci);
      const uint32_t oh = ok ? static_cast<uint32_t>(ch) * cs + static_cast<uint32_t>(gh * a.W + gw) * 2u : OOB;
      hv[hh] = __builtin_amdgcn_raw_buffer_load_b16(rs, oh, 0, 0);
    }
  };

  // transpose the staged registers into LDS buffer `buf`; the designated
  // workgroup also writes its interior rows of a cache frame to cache_out
  auto store_stage = [&](int s, int buf) {
    unsigned char* tile = lds + buf * BUF;
    const int k = k_lo + s % ntap, c0 = (s / ntap) * BKC;
    const int f = o + k * a.dt - a.p_l;
    const bool cw = a.write_cache && s < nst && ct == 0 && f >= a.Z - a.L &&
                    (k == a.Kt - 1 || o < a.dt);
#pragma unroll
    for (int tt = 0; tt < TPT; ++tt) {
      const int t = tid + tt * NT;
      int g, rr, q;
      task(t, g, rr, q);
      if (t < NTASK && rr < TH) {
        u32x4 pr[8];
        transpose8x8(sv[tt], pr);
#pragma unroll
        for (int p = 0; p < 8; ++p)
          *reinterpret_cast<u32x4*>(tile + (rr * TW + 1 + 8 * q + p) * PIXB + 16 * g) = pr[p];
        const int gh = h0 - 1 + rr, w = w0 + 8 * q;
        if (cw && rr >= 1 && rr <= BH && gh < a.H && w < a.W) {
          const int fo = f - (a.Z - a.L);
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int c = c0 + 8 * g + j;
            if (c >= a.Ci) break;
            uint16_t* dst = a.cache_out +
                            ((static_cast<int64_t>(n) * a.Ci + c) * a.L + fo) * a.hw +
                            static_cast<int64_t>(gh) * a.W + w;
            if (ALIGNED) {
              *reinterpret_cast<u32x4*>(dst) = sv[tt][j];
            } else {
#pragma unroll
              for (int e = 0; e < 8; ++e)
                if (w + e < a.W) dst[e] = static_cast<uint16_t>(sv[tt][j][e >> 1] >> (16 * (e & 1)));
            }
          }
        }
      }
    }
#pragma unroll
    for (int hh = 0; hh < HPT; ++hh) {
      const int e = tid + hh * NT;
      if (e < NHALO) {
        const int ch = e % BKC, side = (e / BKC) % 2, rr = e / (2 * BKC);
        *reinterpret_cast<uint16_t*>(tile + (rr * TW + (side ? TW - 1 : 0)) * PIXB + 2 * ch) = hv[hh];
      }
    }
  };

  // Weights of step (stage s, spatial offset ij) for this wave's fragments.
  // The fragment index is clamped to the last packed fragment: past Co it
  // only feeds accumulator rows that are never stored, and for the stage
  // after the last one (prefetched, never used) it keeps the address inside
  // the packed weights.
  u32x4 wr[3][WCO];
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<u32x4*>(a.wpack), 0, static_cast<int>(a.wpack_bytes), 0x00020000);
  const uint32_t wlane = static_cast<uint32_t>(lane) * 16u;
  const uint32_t nfrag = a.wpack_bytes / 1024u;
  auto load_w = [&](int s, int ij, u32x4 (&dst)[WCO]) {
    const int k = k_lo + s % ntap, chunk = s / ntap;
    const uint32_t row = static_cast<uint32_t>((k * 9 + ij) * a.chunks + chunk) *
                         static_cast<uint32_t>(a.cofrags);
#pragma unroll
    for (int cf = 0; cf < WCO; ++cf) {
      const uint32_t frag = min(row + static_cast<uint32_t>(min(cofrag0 + cf, a.cofrags - 1)), nfrag - 1);
      dst[cf] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(wrs, wlane, frag * 1024u, 0));
    }
  };

  f32x4 acc[WCO][NPF];
#pragma unroll
  for (int i = 0; i < WCO; ++i)
#pragma unroll
    for (int j = 0; j < NPF; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // per-lane LDS offset of this wave's B operand (pixel l % 16, channel group l / 16)
  const int lane_off = (wpx * WR * TW + (lane & 15)) * PIXB + (lane >> 4) * 16;

  if (nst > 0) {
    load_w(0, 0, wr[0]);
    load_w(0, 1, wr[1]);
    for (int part = 0; part < 5; ++part) load_stage(0, part);
    store_stage(0, 0);
    __syncthreads();
  }

  // B fragments of one (kh, kw) step for this wave
  auto load_b = [&](const unsigned char* tile, int ij, u32x4 (&dst)[NPF]) {
    const int ki = ij / 3, kj = ij % 3;
#pragma unroll
    for (int pf = 0; pf < NPF; ++pf) {
      const int rp = pf / WCF, cfb = pf % WCF;
      dst[pf] = *reinterpret_cast<const u32x4*>(tile + ((rp + ki) * TW + cfb * 16 + kj) * PIXB);
    }
  };

  // Step order inside a stage: the B fragments of the next (kh, kw) step and
  // the weights two steps ahead are issued between this step's MFMAs (an
  // explicit interleave), so the matrix pipe is not left idle while loads
  // issue.  Loads for a stage past the last one are issued anyway and read
  // zeros (out-of-range offsets): keeping them unconditional keeps the step
  // one basic block that the interleave can schedule.
  u32x4 bv[2][NPF];
  for (int s = 0; s < nst; ++s) {
    const unsigned char* tile = lds + (s & 1) * BUF + lane_off;
    load_b(tile, 0, bv[0]);
#pragma unroll
    for (int ij = 0; ij < 9; ++ij) {
      // One fresh LDS read per fragment and step: the rows of neighbouring
      // kh offsets overlap, and keeping them live across steps would cost
      // more registers than the LDS bandwidth it saves.
      asm volatile("" ::: "memory");
      __builtin_amdgcn_sched_barrier(0);
      if (ij + 1 < 9) load_b(tile, ij + 1, bv[(ij + 1) & 1]);
      load_w(s + (ij + 2) / 9, (ij + 2) % 9, wr[(ij + 2) % 3]);
      if (ij < 5) load_stage(s + 1, ij);
      // The other LDS buffer was last read in stage s - 1, which every wave
      // has finished (barrier below), so the next stage's tile is written
      // here, mid-stage, interleaved with this stage's matrix-core work.
      if (ij == 7) store_stage(s + 1, (s + 1) & 1);
#pragma unroll
      for (int pf = 0; pf < NPF; ++pf)
#pragma unroll
        for (int cf = 0; cf < WCO; ++cf)
          acc[cf][pf] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(bf16x8, bv[ij & 1][pf]), __builtin_bit_cast(bf16x8, wr[ij % 3][cf]),
              acc[cf][pf], 0, 0, 0);
      // interleave: LDS reads, then global reads, then LDS writes, each
      // between pairs of MFMAs (masks: 0x008 MFMA, 0x100 DS read,
      // 0x020 VMEM read, 0x200 DS write)
      if (ij + 1 < 9)
        for (int q = 0; q < NPF; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
      for (int q = 0; q < WCO + (ij < 4 ? TPT * 2 : ij == 4 ? HPT : 0); ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      }
      if (ij == 7)
        for (int q = 0; q < TPT * 8 + HPT; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
        }
    }
    __syncthreads();
  }

  // ---- epilogue: bias once, round to bf16, NCTHW store.  With the
  // activations as the A operand, lane l holds output channel l % 16 for the
  // four consecutive pixels 4 * (l / 16) .. + 3 of each fragment: one 8-byte
  // store per fragment.
  const int64_t plane = static_cast<int64_t>(a.To) * a.hw;
  uint16_t* ybase = a.y + (static_cast<int64_t>(n) * a.Co) * plane + static_cast<int64_t>(o) * a.hw;
#pragma unroll
  for (int cf = 0; cf < WCO; ++cf) {
    const int co = (cofrag0 + cf) * 16 + (lane & 15);
    const float bb = (a.has_bias && co < a.Co) ? __uint_as_float(static_cast<uint32_t>(a.bias[co]) << 16) : 0.f;
#pragma unroll
    for (int pf = 0; pf < NPF; ++pf) {
      const int h = h0 + wpx * WR + pf / WCF, w = w0 + (pf % WCF) * 16 + 4 * (lane >> 4);
      if (co >= a.Co || h >= a.H || w >= a.W) continue;
      uint16_t v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = f32_to_bf16(acc[cf][pf][r] + bb);
      uint16_t* dst = ybase + co * plane + static_cast<int64_t>(h) * a.W + w;
      if (ALIGNED && w + 4 <= a.W) {
        *reinterpret_cast<uint2*>(dst) = make_uint2(v[0] | (static_cast<uint32_t>(v[1]) << 16),
                                                   v[2] | (static_cast<uint32_t>(v[3]) << 16));
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (w + r < a.W) dst[r] = v[r];
      }
    }
  }
}

template <int WCO, int WR, int WCF, int WAVES_CO, int WAVES_PX>
hipError_t run(const Geo& g, Args a, bool aligned, hipStream_t s) {
  constexpr int BCO = 16 * WCO * WAVES_CO, BH = WR * WAVES_PX, BW = 16 * WCF;
  a.tiles_co = static_cast<int>((g.d.Co + BCO - 1) / BCO);
  a.tiles_w = static_cast<int>((g.Wo + BW - 1) / BW);
  a.tiles_h = static_cast<int>((g.Ho + BH - 1) / BH);
  const int64_t blocks = static_cast<int64_t>(a.tiles_co) * a.tiles_w * a.tiles_h * g.To * g.d.N;
  if (blocks == 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  a.nblocks = static_cast<int>(blocks);
  const dim3 grid(static_cast<unsigned>(blocks)), block(64 * WAVES_CO * WAVES_PX);
  if (aligned)
    hipLaunchKernelGGL((conv3d_bf16<WCO, WR, WCF, WAVES_CO, WAVES_PX, true>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((conv3d_bf16<WCO, WR, WCF, WAVES_CO, WAVES_PX, false>), grid, block, 0, s, a);
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

hipError_t launch_fast_bf16(const Geo& g, const void* x, const void* cache, const void* wpack,
                            const void* bias, void* y, void* cache_out, bool* cache_written,
                            hipStream_t s) {
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
  // 32-bit buffer offsets: one 32-channel chunk of a source frame and the
  // packed weights must each span less than 2 GiB
  const int64_t frames = g.d.T > g.d.Tc ? g.d.T : g.d.Tc;
  if (static_cast<int64_t>(BKC) * frames * a.hw * 2 >= 0x7fffffff || p.elems() * 2 >= 0x7fffffff)
    return hipErrorInvalidValue;
  a.has_bias = g.d.has_bias ? 1 : 0;
  a.write_cache = (g.L > 0 && cache_covered(g)) ? 1 : 0;
  *cache_written = a.write_cache != 0;
  const bool aligned = (g.d.W % 8 == 0) && (x == nullptr || aligned16(x)) &&
                       (cache == nullptr || aligned16(cache)) &&
                       (cache_out == nullptr || aligned16(cache_out));
  const int64_t Co = g.d.Co;
  if (Co > 128 && Co % 192 == 0) return run<6, 2, 4, 2, 2>(g, a, aligned, s);
  if (Co <= 96) return run<6, 2, 4, 1, 4>(g, a, aligned, s);
  return run<5, 2, 4, 2, 2>(g, a, aligned, s);
}

}  // namespace c3c
