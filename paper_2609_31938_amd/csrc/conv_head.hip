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
// one workgroup per compute unit).  A stage's [32 ch][512 px] window tile
// is copied into LDS as it lies in memory and read back with the
// transposing ds_read_b64_tr_b16 (the A operand: 8 channels of one pixel per
// lane); the B operand for column n = 9-tap index ij times Co plus co is the
// 16-byte lane slot of the packed 3x3 weights' fragment (tap k*9 + ij,
// chunk, 0) that holds output channel co, so the fast route's one weight
// packing serves this kernel too.  Two-stage pipeline with one barrier per
// stage.  After a group's last stage, each of its output frames' accumulators
// go to LDS as D[n][px] in fp32 in turn, and the workgroup sums the nine
// shifted D values of each output, adds the bias once and rounds once.
// A frame of the new cache is written from the staging registers by the
// group that first stages it (its interior segments: each element has one
// writer), so the caller copies no cache when every cache frame is staged.
//
// Measured on the 96 -> 3 480x832 layer (5 chunks): the same 0.24-0.25 ms
// as the earlier per-output-frame form (with its separate cache copy), with
// half the window traffic; three register sets of staged windows (two
// stages of load latency) measured the same as two.
//
// Requires W a multiple of 8, 16-byte-aligned x / cache, 8-byte-aligned y
// (and a 16-byte-aligned cache_out for the fused cache write).
#include <algorithm>

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
  uint16_t* cache_out;
  int64_t hw;
  int N, Ci, Co, T, Tc, H, W, To, Z, dt, p_l, Kt, L;
  int chunks, cofrags, tiles_w, tiles_h, nblocks;
  uint32_t wpack_bytes;
  int has_bias, write_cache;
};

// OG output frames per pass (a group); NF 16-column fragments of D per tap.
template <int NF, int OG>
__global__ __launch_bounds__(256, 1) void conv_head(HeadArgs a) {
  __shared__ __align__(16) unsigned char lds[lds_bytes(NF)];
  constexpr uint32_t OOB = 0x80000000u;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

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
  const int64_t cs_c = static_cast<int64_t>(a.Tc) * a.hw, cs_x = static_cast<int64_t>(a.T) * a.hw;

  // staging: segment q = tid + 256 i -> channel q / 64, window row (q % 64) / 8,
  // columns 8 (q % 8) .. + 7; outside the image an out-of-range offset (zeros;
  // W is a multiple of 8, so a segment is wholly inside or outside).  s_in:
  // the segment lies in this tile's output rows and columns (the part of the
  // window the new cache takes from this workgroup)
  uint32_t s_ch[HSPT], s_px[HSPT], s_lds[HSPT];
  bool s_in[HSPT];
#pragma unroll
  for (int i = 0; i < HSPT; ++i) {
    const int q = tid + 256 * i, ch = q / (HPX / 8), rem = q % (HPX / 8);
    const int r = rem / (HC / 8), sg = rem % (HC / 8);
    const int gh = wh0 + r, gw = ww0 + 8 * sg;
    const bool ok = gh >= 0 && gh < a.H && gw >= 0 && gw < a.W;
    s_ch[i] = static_cast<uint32_t>(ch);
    s_px[i] = ok ? static_cast<uint32_t>(gh * a.W + gw) * 2u : OOB;
    s_lds[i] = static_cast<uint32_t>(hrow(ch) + (r * HC + 8 * sg) * 2);
    s_in[i] = ok && r >= 1 && r <= OR && sg >= 1 && sg <= OC / 8;
  }

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

  f32x4 acc[OG][NF][HPF];
  float* D = reinterpret_cast<float*>(lds);
  const int64_t plane = static_cast<int64_t>(a.To) * a.hw;
  int f_done = -1;  // the last source frame staged by an earlier group

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
    const int padded = (nst + 1) & ~1;

#pragma unroll
    for (int u = 0; u < OG; ++u)
#pragma unroll
      for (int q = 0; q < NF; ++q)
#pragma unroll
        for (int pf = 0; pf < HPF; ++pf) acc[u][q][pf] = f32x4{0.f, 0.f, 0.f, 0.f};

    // stages in order: (af, ac) = frame and chunk of the next one to load;
    // (wf, wc) the same for the next weights.  The resource of a stage starts
    // at channel 32 ac of frame af and ends after the last real channel's
    // plane (channels past Ci read 0); empty past the last stage.
    int af = f_lo, ac = 0, wf = f_lo, wc = 0;
    auto next_rsrc = [&](uint32_t& cs, int& fr, int& c0) {
      const bool real = af <= f_hi;
      c0 = ac * HK;
      fr = af;
      const bool in_cache = af < a.Tc;
      const int64_t cstride = in_cache ? cs_c : cs_x;
      const uint16_t* base = in_cache ? a.cache : a.x;
      const int64_t off = real ? static_cast<int64_t>(in_cache ? af : af - a.Tc) * a.hw +
                                     (static_cast<int64_t>(n) * a.Ci + c0) * cstride
                               : 0;
      int64_t bytes = ((a.Ci - 1 - c0) * cstride + a.hw) * 2;
      if (!real || bytes < 0) bytes = 0;
      if (bytes > 0x7fffffff) bytes = 0x7fffffff;
      cs = static_cast<uint32_t>(cstride * 2);
      if (++ac == a.chunks) {
        ac = 0;
        ++af;
      }
      return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base + off), 0,
                                               static_cast<int>(bytes), 0x00020000);
    };
    // Where a stage's frame goes in the new cache: a frame of the new cache
    // staged for the first time (workgroup-uniform) has its interior segments
    // written to cache_out, when the staged values are stored to LDS, through
    // a resource that ends after the last real channel.
    struct CacheDst {
      __amdgpu_buffer_rsrc_t rs;
      uint32_t cs;
      bool on;
    };
    const uint32_t ccs = static_cast<uint32_t>(static_cast<int64_t>(a.L) * a.hw * 2);
    // the activations of the next stage
    auto load_act = [&](u32x4 (&v)[HSPT], CacheDst& cd) {
      uint32_t cs;
      int fr, c0;
      const __amdgpu_buffer_rsrc_t rs = next_rsrc(cs, fr, c0);
#pragma unroll
      for (int i = 0; i < HSPT; ++i)
        v[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                             rs, s_px[i] == OOB ? OOB : s_ch[i] * cs + s_px[i], 0, 0));
      cd.on = a.write_cache && fr <= f_hi && fr > f_done && fr >= a.Z - a.L;
      const int64_t cl = static_cast<int64_t>(a.L) * a.hw;
      uint16_t* cb = a.cache_out + (cd.on ? (static_cast<int64_t>(n) * a.Ci + c0) * cl +
                                                static_cast<int64_t>(fr - (a.Z - a.L)) * a.hw
                                          : 0);
      int64_t cbytes = ((a.Ci - 1 - c0) * cl + a.hw) * 2;
      if (!cd.on || cbytes < 0) cbytes = 0;
      if (cbytes > 0x7fffffff) cbytes = 0x7fffffff;
      cd.rs = __builtin_amdgcn_make_buffer_rsrc(cb, 0, static_cast<int>(cbytes), 0x00020000);
    };
    // the weights of the next stage for each output frame of the group: tap
    // k = (f + p_l - o) / d_t when that is a whole tap index, else zeros (and
    // the frame's products are skipped: tap_ok)
    auto load_w = [&](u32x4 (&v)[OG][NF], bool (&ok)[OG]) {
      const bool real = wf <= f_hi;
#pragma unroll
      for (int u = 0; u < OG; ++u) {
        const int o = og0 + u, kd = wf + a.p_l - o;
        const int k = kd >= 0 ? kd / a.dt : -1;
        ok[u] = real && o < og1 && kd >= 0 && kd % a.dt == 0 && k < a.Kt;
        const uint32_t base = static_cast<uint32_t>((ok[u] ? k : 0) * 9 * a.chunks + wc) * frag_bytes;
#pragma unroll
        for (int q = 0; q < NF; ++q)
          v[u][q] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                  wrs, ok[u] && w_ok[q] ? base + w_off[q] : OOB, 0, 0));
      }
      if (++wc == a.chunks) {
        wc = 0;
        ++wf;
      }
    };
    auto store_act = [&](const u32x4 (&v)[HSPT], const CacheDst& cd, int buf) {
#pragma unroll
      for (int i = 0; i < HSPT; ++i) *reinterpret_cast<u32x4*>(lds + buf * HBUF + s_lds[i]) = v[i];
      if (cd.on) {
#pragma unroll
        for (int i = 0; i < HSPT; ++i)
          __builtin_amdgcn_raw_buffer_store_b128(v[i], cd.rs, s_in[i] ? s_ch[i] * ccs + s_px[i] : OOB,
                                                 0, 0);
      }
    };

    u32x4 act0[HSPT], act1[HSPT];
    CacheDst cd0, cd1;
    u32x4 w0v[OG][NF], w1v[OG][NF];
    bool ok0[OG], ok1[OG];
    load_w(w0v, ok0);
    load_act(act0, cd0);
    load_act(act1, cd1);
    store_act(act0, cd0, 0);
    __syncthreads();

    // one stage: weights of s + 1 and activations of s + 2 issued, the
    // products of s for every output frame it feeds, then s + 1's
    // activations into the other buffer (last read in stage s - 1, before
    // its barrier)
    auto stage = [&](int buf, const u32x4 (&w_cur)[OG][NF], const bool (&ok_cur)[OG],
                     u32x4 (&w_nxt)[OG][NF], bool (&ok_nxt)[OG], u32x4 (&a_free)[HSPT],
                     CacheDst& c_free, const u32x4 (&a_next)[HSPT], const CacheDst& c_next) {
      load_w(w_nxt, ok_nxt);
      load_act(a_free, c_free);
      i16x8 av[HPF];
#pragma unroll
      for (int pf = 0; pf < HPF; ++pf) av[pf] = read_a(buf, pf);
#pragma unroll
      for (int u = 0; u < OG; ++u) {
        if (!ok_cur[u]) continue;  // workgroup-uniform
#pragma unroll
        for (int pf = 0; pf < HPF; ++pf)
#pragma unroll
          for (int q = 0; q < NF; ++q)
            acc[u][q][pf] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, av[pf]), __builtin_bit_cast(bf16x8, w_cur[u][q]), acc[u][q][pf],
                0, 0, 0);
      }
      store_act(a_next, c_next, buf ^ 1);
      __syncthreads();
    };
    for (int s = 0; s < padded; s += 2) {
      stage(0, w0v, ok0, w1v, ok1, act0, cd0, act1, cd1);
      stage(1, w1v, ok1, w0v, ok0, act1, cd1, act0, cd0);
    }
    f_done = f_hi;

    // per output frame of the group: D[n][window pixel] in fp32 over the
    // stage buffers (lane l holds pixels 4 (l / 16) .. + 3 of column
    // 16 q + l % 16 of each fragment), then the gather: output (co, row r,
    // columns 4 c4 .. + 3) sums D[(i j) Co + co] at window row r + i, window
    // columns 7 + 4 c4 + j .. + 3; bias once, one round-to-nearest-even,
    // 8-byte NCTHW store
#pragma unroll
    for (int u = 0; u < OG; ++u) {
      const int o = og0 + u;
      if (o >= og1) break;
#pragma unroll
      for (int q = 0; q < NF; ++q) {
        const int col = 16 * q + (lane & 15);
        if (col >= 9 * a.Co) continue;
#pragma unroll
        for (int pf = 0; pf < HPF; ++pf) {
          const int px = (2 * wave + pf / (HC / 16)) * HC + (pf % (HC / 16)) * 16 + 4 * g;
          *reinterpret_cast<f32x4*>(D + col * DPITCH + px) = acc[u][q][pf];
        }
      }
      __syncthreads();
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
      __syncthreads();  // D is rewritten by the next frame, the stage buffers by the next group
    }
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
  const dim3 grid(static_cast<unsigned>(blocks)), block(256);
  // output frames per group: 4 (the 256 accumulator registers of 4 frames x
  // 2 fragments x 8 pixel fragments), 2 with three column fragments
  if (nf == 1)
    hipLaunchKernelGGL((conv_head<1, 4>), grid, block, 0, s, a);
  else if (nf == 2)
    hipLaunchKernelGGL((conv_head<2, 4>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((conv_head<3, 2>), grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace c3c
