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
// Workgroup = 6 output rows x 48 output columns of one (n, o) frame, from
// an input window of 8 rows x 64 columns (origin one row above and eight
// columns left of the output tile, so that every 16-byte row segment of the
// window is aligned).  4 waves, wave v owning window rows 2v, 2v + 1: 8
// pixel fragments x NF column fragments of accumulators.  The window is
// sized so that two workgroups fit a compute unit for Co <= 3 (NF = 2: 67 KB
// of LDS, at most 128 registers a lane; the NF = 3 instance for Co = 4, 5
// needs 92.9 KB for its D rows and runs one workgroup per unit): a stage is
// short (16 products per wave), and
// the second workgroup's stages cover the first's memory waits (measured: 8 x
// 80 windows at one workgroup per unit were 1.3x slower, 8 x 48 at three
// 1.1x slower).  A stage is one active tap and one 32-channel chunk: its
// [32 ch][512 px] window tile is
// copied into LDS as it lies in memory and read back with the transposing
// ds_read_b64_tr_b16 (the A operand: 8 channels of one pixel per lane); the
// B operand for column n = 9-tap index ij times Co plus co is the 16-byte
// lane slot of the packed 3x3 weights' fragment (tap k*9 + ij, chunk, 0) that
// holds output channel co, so the fast route's one weight packing serves
// this kernel too.  Two-stage pipeline with one barrier per stage as in the
// 1x1 kernel.  After the last stage the accumulators go to LDS as D[n][px]
// in fp32, and the workgroup sums the nine shifted D values of each output,
// adds the bias once and rounds once.
//
// Requires W a multiple of 8, 16-byte-aligned x / cache, 8-byte-aligned y.
// The new cache is copied by the caller.
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

constexpr int HK = 32;                 // input channels per stage
constexpr int HR = 8, HC = 64;         // input window rows x columns
constexpr int OR = 6, OC = 48;         // output rows x columns per workgroup
constexpr int HPX = HR * HC;           // window pixels
constexpr int HPF = 2 * (HC / 16);     // pixel fragments per wave (2 rows)
// LDS offset of staged channel row c: 1024 B + 32 B, and 128 B more after
// every 8 channels.  The 32 lanes one transposing read serves per cycle take
// 32 B from each of channels {0..3, 8..11} (+4, +16, +20 for the other
// halves): banks 0, 8, 16, 24 and 32, 40, 48, 56, disjoint 8-bank groups.
constexpr int HPITCH = HPX * 2 + 32;
constexpr int hrow(int c) { return c * HPITCH + (c >> 3) * 128; }
constexpr int HBUF = hrow(HK);
constexpr int HSEG = HK * HPX / 8;     // 16-byte segments of a stage tile
constexpr int HSPT = HSEG / 256;       // per thread
static_assert(HSEG % 256 == 0, "the stage tile splits evenly over the threads");
constexpr int max_co(int nf) { return 16 * nf / 9; }
// D rows (one per column n) of the window's 512 pixels, 516 floats apart: the
// 16 lanes of a fragment row write 16 consecutive n with 16-byte stores, and
// 516 = 4 mod 64 banks puts them in 16 disjoint 4-bank groups
constexpr int DPITCH = HPX + 4;
constexpr int lds_bytes(int nf) {
  return 2 * HBUF > 9 * max_co(nf) * DPITCH * 4 ? 2 * HBUF : 9 * max_co(nf) * DPITCH * 4;
}

struct HeadArgs {
  const uint16_t* x;
  const uint16_t* cache;
  const u32x4* wpack;
  const uint16_t* bias;
  uint16_t* y;
  int64_t hw;
  int N, Ci, Co, T, Tc, H, W, To, Z, dt, p_l, Kt;
  int chunks, cofrags, tiles_w, tiles_h, nblocks;
  uint32_t wpack_bytes;
  int has_bias;
};

template <int NF>
__global__ __launch_bounds__(256, 2) void conv_head(HeadArgs a) {
  __shared__ __align__(16) unsigned char lds[lds_bytes(NF)];
  constexpr uint32_t OOB = 0x80000000u;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  // workgroups numbered so that each XCD runs a contiguous range: the output
  // frames of one spatial tile (which share source frames) run together
  int b;
  {
    const int per = a.nblocks / 8, rem = a.nblocks % 8;
    const int xcd = static_cast<int>(blockIdx.x) % 8, slot = static_cast<int>(blockIdx.x) / 8;
    b = (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + slot;
  }
  const int o = b % a.To;
  b /= a.To;
  const int tw = b % a.tiles_w;
  b /= a.tiles_w;
  const int th = b % a.tiles_h;
  const int n = b / a.tiles_h;
  const int h0 = th * OR, w0 = tw * OC;
  const int wh0 = h0 - 1, ww0 = w0 - 8;  // window origin

  // active taps (Eq. 4): source frame o + k dt - p_l in [0, Z)
  int k_lo = 0;
  while (k_lo < a.Kt && o + k_lo * a.dt - a.p_l < 0) ++k_lo;
  int k_hi = a.Kt - 1;
  while (k_hi >= 0 && o + k_hi * a.dt - a.p_l >= a.Z) --k_hi;
  const int ntap = k_hi >= k_lo ? k_hi - k_lo + 1 : 0;
  const int nst = ntap * a.chunks;
  const int padded = (nst + 1) & ~1;

  // activation stages in order: (ak, ac) = tap and chunk of the next one; its
  // resource starts at channel 32 ac of frame f and ends after the last real
  // channel's plane (channels past Ci read 0), empty past the last stage
  const int64_t cs_c = static_cast<int64_t>(a.Tc) * a.hw, cs_x = static_cast<int64_t>(a.T) * a.hw;
  int ak = k_lo, ac = 0;
  auto next_rsrc = [&](uint32_t& cs) {
    const bool real = ak <= k_hi;
    const int c0 = ac * HK;
    const int f = o + ak * a.dt - a.p_l;
    const bool in_cache = f < a.Tc;
    const int64_t cstride = in_cache ? cs_c : cs_x;
    const uint16_t* base = in_cache ? a.cache : a.x;
    const int64_t off = static_cast<int64_t>(in_cache ? f : f - a.Tc) * a.hw +
                        (static_cast<int64_t>(n) * a.Ci + c0) * cstride;
    int64_t bytes = ((a.Ci - 1 - c0) * cstride + a.hw) * 2;
    if (!real || bytes < 0) bytes = 0;
    if (bytes > 0x7fffffff) bytes = 0x7fffffff;
    cs = static_cast<uint32_t>(cstride * 2);
    if (++ac == a.chunks) {
      ac = 0;
      ++ak;
    }
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(real ? base + off : base), 0,
                                             static_cast<int>(bytes), 0x00020000);
  };

  // staging: segment q = tid + 256 i -> channel q / 64, window row (q % 64) / 8,
  // columns 8 (q % 8) .. + 7; outside the image an out-of-range offset (zeros;
  // W is a multiple of 8, so a segment is wholly inside or outside)
  uint32_t s_ch[HSPT], s_px[HSPT], s_lds[HSPT];
#pragma unroll
  for (int i = 0; i < HSPT; ++i) {
    const int q = tid + 256 * i, ch = q / (HPX / 8), rem = q % (HPX / 8);
    const int r = rem / (HC / 8), sg = rem % (HC / 8);
    const int gh = wh0 + r, gw = ww0 + 8 * sg;
    const bool ok = gh >= 0 && gh < a.H && gw >= 0 && gw < a.W;
    s_ch[i] = static_cast<uint32_t>(ch);
    s_px[i] = ok ? static_cast<uint32_t>(gh * a.W + gw) * 2u : OOB;
    s_lds[i] = static_cast<uint32_t>(hrow(ch) + (r * HC + 8 * sg) * 2);
  }
  auto load_act = [&](u32x4 (&v)[HSPT]) {
    uint32_t cs;
    const __amdgpu_buffer_rsrc_t rs = next_rsrc(cs);
#pragma unroll
    for (int i = 0; i < HSPT; ++i)
      v[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                           rs, s_px[i] == OOB ? OOB : s_ch[i] * cs + s_px[i], 0, 0));
  };
  auto store_act = [&](const u32x4 (&v)[HSPT], int buf) {
#pragma unroll
    for (int i = 0; i < HSPT; ++i) *reinterpret_cast<u32x4*>(lds + buf * HBUF + s_lds[i]) = v[i];
  };

  // weights: column n = 16 q + lane % 16 is (ij = n / Co, co = n % Co) for
  // n < 9 Co; its 8 channels are the lane slot co + 16 (lane / 16) of packed
  // fragment (tap k 9 + ij, chunk, output fragment 0); other columns are zero
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<u32x4*>(a.wpack), 0, static_cast<int>(a.wpack_bytes), 0x00020000);
  const uint32_t frag_bytes = static_cast<uint32_t>(a.cofrags) * 1024u;
  uint32_t w_off[NF];
  bool w_ok[NF];
#pragma unroll
  for (int q = 0; q < NF; ++q) {
    const int col = 16 * q + (lane & 15);
    w_ok[q] = col < 9 * a.Co;
    const int ij = w_ok[q] ? col / a.Co : 0, co = w_ok[q] ? col % a.Co : 0;
    w_off[q] = static_cast<uint32_t>(ij * a.chunks) * frag_bytes +
               static_cast<uint32_t>(co + 16 * (lane >> 4)) * 16u;
  }
  // weight stages in order: (wk, wc) = tap and chunk of the next one, its
  // packed row (wk 9 chunks + wc) advanced without a division
  int wk = k_lo, wc = 0;
  uint32_t wbase = static_cast<uint32_t>(k_lo * 9 * a.chunks) * frag_bytes;
  auto load_w = [&](u32x4 (&v)[NF]) {
    const bool real = wk <= k_hi;
#pragma unroll
    for (int q = 0; q < NF; ++q)
      v[q] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                           wrs, real && w_ok[q] ? wbase + w_off[q] : OOB, 0, 0));
    wbase += frag_bytes;
    if (++wc == a.chunks) {  // next tap: 8 more (kh, kw) rows of chunks
      wc = 0;
      ++wk;
      wbase += static_cast<uint32_t>(8 * a.chunks) * frag_bytes;
    }
  };

  // transposing operand read of pixel fragment pf of this wave (window row
  // 2 wave + pf / (HC / 16), columns 16 (pf % (HC / 16)) ..): lane j of 16-lane block g names
  // channel 8g + 4h + j / 4 at pixel group 4 (j % 4)
  const int j = lane & 15, g = lane >> 4;
  const int ra = hrow(8 * g + (j >> 2)) + (2 * wave * HC + 4 * (j & 3)) * 2;
  auto read_a = [&](int buf, int pf) {
    const unsigned char* p = lds + buf * HBUF + ra + ((pf / (HC / 16)) * HC + (pf % (HC / 16)) * 16) * 2;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 4 * HPITCH));
    return i16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  };

  f32x4 acc[NF][HPF];
#pragma unroll
  for (int q = 0; q < NF; ++q)
#pragma unroll
    for (int pf = 0; pf < HPF; ++pf) acc[q][pf] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 act0[HSPT], act1[HSPT];
  u32x4 w0v[NF], w1v[NF];
  load_w(w0v);
  load_act(act0);
  load_act(act1);
  store_act(act0, 0);
  __syncthreads();

  // one stage: weights of s + 1 and activations of s + 2 issued, the
  // products of s, then s + 1's activations into the other buffer (last read
  // in stage s - 1, before its barrier)
  auto stage = [&](int s, int buf, const u32x4 (&w_cur)[NF], u32x4 (&w_nxt)[NF], u32x4 (&a_free)[HSPT],
                   const u32x4 (&a_next)[HSPT]) {
    load_w(w_nxt);
    load_act(a_free);
    i16x8 av[HPF];
#pragma unroll
    for (int pf = 0; pf < HPF; ++pf) av[pf] = read_a(buf, pf);
#pragma unroll
    for (int pf = 0; pf < HPF; ++pf)
#pragma unroll
      for (int q = 0; q < NF; ++q)
        acc[q][pf] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            __builtin_bit_cast(bf16x8, av[pf]), __builtin_bit_cast(bf16x8, w_cur[q]), acc[q][pf], 0, 0, 0);
    store_act(a_next, buf ^ 1);
    __syncthreads();
  };
  for (int s = 0; s < padded; s += 2) {
    stage(s, 0, w0v, w1v, act0, act1);
    stage(s + 1, 1, w1v, w0v, act1, act0);
  }

  // D[n][window pixel] in fp32 over the stage buffers (the last stage's
  // barrier has passed): lane l holds pixels 4 (l / 16) .. + 3 of column
  // 16 q + l % 16 of each fragment
  float* D = reinterpret_cast<float*>(lds);
#pragma unroll
  for (int q = 0; q < NF; ++q) {
    const int col = 16 * q + (lane & 15);
    if (col >= 9 * a.Co) continue;
#pragma unroll
    for (int pf = 0; pf < HPF; ++pf) {
      const int px = (2 * wave + pf / (HC / 16)) * HC + (pf % (HC / 16)) * 16 + 4 * g;
      *reinterpret_cast<f32x4*>(D + col * DPITCH + px) = acc[q][pf];
    }
  }
  __syncthreads();

  // gather: output (co, row r, columns 4 c4 .. + 3) sums D[(i j) Co + co] at
  // window row r + i, window columns 7 + 4 c4 + j .. + 3; bias once, one
  // round-to-nearest-even, 8-byte NCTHW store
  const int64_t plane = static_cast<int64_t>(a.To) * a.hw;
  for (int t = tid; t < a.Co * OR * (OC / 4); t += 256) {
    const int co = t / (OR * (OC / 4)), rem = t % (OR * (OC / 4));
    const int r = rem / (OC / 4), c4 = rem % (OC / 4);
    const int h = h0 + r, w = w0 + 4 * c4;
    if (h >= a.H || w >= a.W) continue;
    const float bb = a.has_bias ? __uint_as_float(static_cast<uint32_t>(a.bias[co]) << 16) : 0.f;
    float s4[4] = {bb, bb, bb, bb};
#pragma unroll
    for (int i = 0; i < 3; ++i)
#pragma unroll
      for (int jj = 0; jj < 3; ++jj) {
        const float* src = D + ((i * 3 + jj) * a.Co + co) * DPITCH + (r + i) * HC + 7 + 4 * c4 + jj;
#pragma unroll
        for (int e = 0; e < 4; ++e) s4[e] += src[e];
      }
    const uint32_t v01 = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{s4[0], s4[1]}), bf16x2));
    const uint32_t v23 = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{s4[2], s4[3]}), bf16x2));
    uint16_t* dst = a.y + (static_cast<int64_t>(n) * a.Co + co) * plane + static_cast<int64_t>(o) * a.hw +
                    static_cast<int64_t>(h) * a.W + w;
    *reinterpret_cast<uint2*>(dst) = make_uint2(v01, v23);
  }
}

bool aligned_to(const void* p, uintptr_t m) { return (reinterpret_cast<uintptr_t>(p) & (m - 1)) == 0; }

}  // namespace

bool head_eligible(const Geo& g, const void* x, const void* cache, const void* y) {
  const c3c_conv_desc& d = g.d;
  if (d.Co > max_co(3) || d.W % 8 != 0) return false;
  // buffer offsets are 32-bit: one 32-channel slab of a source frame and the
  // packed weights must fit
  const int64_t frames = d.T > d.Tc ? d.T : d.Tc;
  if (static_cast<int64_t>(HK) * frames * d.H * d.W * 2 >= 0x7fffffff ||
      pack_dims(d).elems() * 2 >= 0x7fffffff)
    return false;
  return aligned_to(x, 16) && (cache == nullptr || aligned_to(cache, 16)) && aligned_to(y, 8);
}

hipError_t launch_head(const Geo& g, const void* x, const void* cache, const void* wpack,
                       const void* bias, void* y, hipStream_t s, LaunchInfo* info) {
  const c3c_conv_desc& d = g.d;
  if (!head_eligible(g, x, cache, y)) return hipErrorInvalidValue;
  const PackDims p = pack_dims(d);
  HeadArgs a;
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
  const int64_t blocks = static_cast<int64_t>(a.tiles_w) * a.tiles_h * g.To * d.N;
  if (info) {
    info->kernel = C3C_KERNEL_HEAD;
    info->tile_co = d.Co;
    info->tile_h = OR;
    info->tile_w = OC;
    info->workgroups = blocks;
    return hipSuccess;
  }
  if (blocks == 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  a.nblocks = static_cast<int>(blocks);
  const int nf = static_cast<int>((9 * d.Co + 15) / 16);
  const dim3 grid(static_cast<unsigned>(blocks)), block(256);
  if (nf == 1)
    hipLaunchKernelGGL(conv_head<1>, grid, block, 0, s, a);
  else if (nf == 2)
    hipLaunchKernelGGL(conv_head<2>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(conv_head<3>, grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace c3c
