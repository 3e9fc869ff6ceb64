// Internal interface between the C-ABI host layer (c3c_host.cpp) and the
// kernel translation units.  Not installed; not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "c3c.h"

namespace c3c {

// Geometry of one validated call (Sec. 4.2: |Z|, p_l, T_o; spatial analogue).
struct Geo {
  c3c_conv_desc d;
  int64_t Z;    // |Z|_T = Tc + T
  int64_t p_l;  // effective left pad = pad_t_base - Tc (may be negative)
  int64_t To, Ho, Wo;
  int64_t L;    // new cache length = min(pad_t_base, |Z|)
  int elem;     // bytes per element
};

// Fast-route packed-weight layout.  The K index of one tap (kt, kh, kw) is the
// input channel; it is cut into chunks of KSTEP channels (16 for bf16, 2 for
// fp32: the K extent of one matrix-core instruction) and the output channels
// into fragments of 32.  Element (tap, chunk, cofrag, lane, e) holds
// w[co = cofrag*32 + lane%32][ci = chunk*KSTEP + (lane/32)*KPL + e][tap],
// zero outside [0, Co) x [0, Ci).
struct PackDims {
  int kpl;        // elements per lane (8 for bf16, 1 for fp32)
  int kstep;      // channels per matrix-core step (2 * kpl)
  int64_t taps;   // Kt * Kh * Kw
  int64_t chunks; // ceil(Ci / kstep)
  int64_t cofrags;// ceil(Co / 32)
  int64_t elems() const { return taps * chunks * cofrags * 64 * kpl; }
};
PackDims pack_dims(const c3c_conv_desc& d);

hipError_t launch_repack(const Geo& g, const void* w, void* wpack, hipStream_t s);
hipError_t launch_unpack(const Geo& g, const void* wpack, void* w, hipStream_t s);
hipError_t launch_fast(const Geo& g, const void* x, const void* cache, const void* wpack,
                       const void* bias, void* y, void* cache_out, hipStream_t s);
hipError_t launch_fallback(const Geo& g, const void* x, const void* cache, const void* w,
                           const void* bias, void* y, hipStream_t s);
hipError_t launch_cache_copy(const Geo& g, const void* x, const void* cache, void* cache_out,
                             hipStream_t s);

}  // namespace c3c
