/*
 * c3c.h -- cached causal Conv3D for AMD Instinct MI355X (gfx950).
 *
 * The library evaluates a cached causal Conv3D call the way the paper's
 * cache-aware lowering defines it (Sec. 4, Eq. 1-4, Alg. 1): every temporal
 * tap k of the kernel is a batched spatial Conv2D over the valid frames of
 * the cache-augmented input Z = [C; X]_T, the taps are summed, the bias is
 * added exactly once, the output is NCTHW, and the cache is replaced by the
 * last frames of Z.  On the fast route all active taps of one call are one
 * implicit-GEMM kernel on bf16 (or fp32) matrix cores with fp32 accumulation;
 * calls the fast route does not support go to a generic direct-Conv3D
 * fallback kernel, and route counters account for every call (Alg. 1 keeps
 * call / fast counters; Sec. 1 and Sec. 6 speak of fallbacks and unsupported
 * cases).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every call returns a status code (enum c3c_status); nothing throws.
 *  - Tensor pointers are DEVICE pointers (HIP device memory) unless stated.
 *    The caller allocates and owns every buffer; the library never allocates
 *    device memory in a compute call.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    Work is enqueued asynchronously on it; the caller synchronises before
 *    reading outputs.  A device fault after enqueue is reported by the HIP
 *    runtime at the next synchronisation, not by the call that enqueued it.
 *  - A c3c_ctx holds the mode bits, the route counters and the histogram of
 *    shapes that went to the fallback.  It is not thread-safe: use one
 *    context per host thread (and, mirroring the paper's attribution of calls
 *    to the active encode or decode scope, one per scope).
 *  - All tensors are contiguous, element type `dtype` throughout:
 *      x         [N][Ci][T][H][W]          the new chunk (X)
 *      cache     [N][Ci][Tc][H][W]         cached prior frames (C); NULL iff Tc == 0
 *      w         [Co][Ci/groups][Kt][Kh][Kw]   the unchanged Conv3D weights
 *      bias      [Co]                      NULL iff has_bias == 0
 *      y         [N][Co][To][Ho][Wo]       output, NCTHW; may be NULL iff To*Ho*Wo*N*Co == 0
 *      cache_out [N][Ci][L][H][W]          the new cache; NULL allowed iff L == 0
 *    where To is Eq. 3 with p_l = pad_t_base - Tc, Ho/Wo the spatial
 *    analogue, and L = min(pad_t_base, Tc + T).
 *  - Size limits (EINVAL beyond them): every size below 2^31, one frame plane
 *    (H*W and Ho*Wo elements) below 2^31 bytes, every tensor below 2^40
 *    elements.
 */
#ifndef C3C_H
#define C3C_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------- status */
typedef enum c3c_status {
  C3C_OK = 0,
  C3C_E_INVAL = 1,       /* null / negative / inconsistent arguments, aliasing */
  C3C_E_UNSUPPORTED = 2, /* strict mode and the call does not route fast      */
  C3C_E_DEVICE = 3,      /* a HIP launch or runtime call failed               */
  C3C_E_INJECTED = 4     /* strict mode and an injected fast-route failure    */
} c3c_status;

/* ---------------------------------------------------------------- dtypes */
typedef enum c3c_dtype {
  C3C_DTYPE_BF16 = 1, /* fast route: bf16 matrix cores, fp32 accumulation   */
  C3C_DTYPE_F32 = 2,  /* fast route: fp32 matrix cores, fp32 accumulation   */
  C3C_DTYPE_F16 = 3   /* fallback route only                               */
} c3c_dtype;

/* ---------------------------------------------------------------- modes */
enum {
  /* an unsupported call or a fast-route failure returns an error instead of
   * falling back (the paper's strict validation mode, Sec. 4.3) */
  C3C_MODE_STRICT = 1u,
  /* every call takes the fallback route: the baseline that must record zero
   * fast hits (acceptance rule, Sec. 5.3) */
  C3C_MODE_FORCE_FALLBACK = 2u,
  /* the fast route fails before launching anything, as a test of the failure
   * path: counted in fast_error, then fallback (or C3C_E_INJECTED if strict) */
  C3C_MODE_INJECT_FAST_FAILURE = 4u,
  /* a bf16 3x3 call that runs unsplit keeps the tile its output-channel count
   * selects even when those tiles fill less than one round of the compute
   * units (by default such a call may take smaller tiles that fill more of
   * them); outputs are bit-identical either way, the accumulation order of
   * every output element being the same: this pins the kernel instance,
   * e.g. to test each tile on small inputs */
  C3C_MODE_CHANNEL_TILES = 8u
};

/* ---------------------------------------------------------------- routes */
typedef enum c3c_route { C3C_ROUTE_FAST = 0, C3C_ROUTE_FALLBACK = 1 } c3c_route;

/* Why a call does not route fast: the first failing clause, tested in this
 * order.  Clauses 2-7 are the paper's guard (Alg. 1), except that clause 4
 * is widened: a 1x1 spatial kernel (a temporal convolution) is accepted at
 * any temporal stride.  Clauses 8-9 state what the fast kernels are
 * specialised for: the 3x3 form (stride 1, pad 1, dilation 1) of the
 * decoder's main convolutions, also with a single temporal tap (a per-frame
 * spatial convolution), and the 1x1 form (stride 1, pad 0) of its temporal
 * convolutions, with at least two temporal taps. */
typedef enum c3c_reason {
  C3C_REASON_NONE = 0,      /* routes fast                                   */
  C3C_REASON_FORCED = 1,    /* C3C_MODE_FORCE_FALLBACK                       */
  C3C_REASON_DTYPE = 2,     /* dtype has no fast kernel (f16)                */
  C3C_REASON_GROUPS = 3,    /* groups != 1                                   */
  C3C_REASON_STRIDE_T = 4,  /* temporal stride != 1, spatial kernel not 1x1 */
  C3C_REASON_PAD_RIGHT = 5, /* pad_t_right < 0                               */
  C3C_REASON_NO_OUTPUT = 6, /* To < 1                                        */
  C3C_REASON_NO_TAP = 7,    /* no (output frame, tap) pair reads a frame of Z */
  C3C_REASON_KT1 = 8,       /* Kt < 2 and the spatial kernel is not the 3x3
                               form (e.g. a 1x1x1 shortcut conv)             */
  C3C_REASON_SPATIAL = 9,   /* spatial kernel is neither 3x3 (stride 1, pad 1,
                               dil 1) nor 1x1 (stride 1, pad 0)              */
  /* not a predicate clause: the call routed fast, the fast route failed and
   * the call fell back (appears only in the fallback-shape histogram) */
  C3C_REASON_FAST_ERROR = 10
} c3c_reason;

/* ---------------------------------------------------------------- descriptor */
/* One Conv3D call (Sec. 4.1 notation).  pad_t_base is p_l^base, the temporal
 * left pad the layer would apply with no cache; the effective left pad is
 * p_l = pad_t_base - Tc (Sec. 4.2) and may be negative, in which case the
 * oldest cache frames are not read.  A causal 3-tap layer has
 * pad_t_base = 2 * dil_t, pad_t_right = 0. */
typedef struct c3c_conv_desc {
  int64_t N, Ci, Co;       /* batch, input / output channels (>= 1)          */
  int64_t T, Tc;           /* new frames, cached frames (>= 0)               */
  int64_t H, W;            /* spatial size (>= 1)                            */
  int64_t Kt, Kh, Kw;      /* kernel size (>= 1)                             */
  int64_t stride_t, stride_h, stride_w; /* >= 1                              */
  int64_t dil_t, dil_h, dil_w;          /* >= 1                              */
  int64_t pad_t_base;      /* p_l^base >= 0                                  */
  int64_t pad_t_right;     /* p_r (any sign; < 0 routes to the fallback)     */
  int64_t pad_h, pad_w;    /* symmetric spatial zero padding (>= 0)          */
  int64_t groups;          /* divides Ci and Co                              */
  int32_t dtype;           /* enum c3c_dtype                                 */
  int32_t has_bias;        /* 0 or 1                                         */
} c3c_conv_desc;

typedef struct c3c_counters {
  /* Invariants: calls = fast + fallback + strict_rejects + failed
   *             fallback = unsupported + forced + fast_error
   * A call is counted in fast / fallback (and its reason) only once its
   * kernels were enqueued without error. */
  uint64_t calls;          /* valid calls (EINVAL calls are not counted)     */
  uint64_t fast;           /* completed on the fast route                    */
  uint64_t fallback;       /* completed on the fallback route                */
  uint64_t unsupported;    /* fell back because a guard clause failed        */
  uint64_t forced;         /* fell back because of C3C_MODE_FORCE_FALLBACK   */
  uint64_t fast_error;     /* fell back because the fast route failed        */
  uint64_t strict_rejects; /* refused in strict mode                         */
  uint64_t repacks;        /* weight repacks enqueued                        */
  uint64_t failed;         /* the fallback's own launch failed: the call
                              returned C3C_E_DEVICE and computed nothing     */
} c3c_counters;

/* One entry of the fallback-shape histogram: the reason and the full call
 * signature (the paper keys runtime signatures by channels, frames, spatial
 * size and cache length, Table 1). */
typedef struct c3c_sig_count {
  int32_t reason;          /* enum c3c_reason */
  int32_t reserved;
  c3c_conv_desc desc;
  uint64_t count;
} c3c_sig_count;

typedef struct c3c_ctx c3c_ctx;

/* ---------------------------------------------------------------- context */
/* Create a context with the given mode bits.  *out receives a host object
 * owned by the caller; free it with c3c_ctx_destroy.  EINVAL if out is NULL
 * or mode has unknown bits. */
int c3c_ctx_create(uint32_t mode, c3c_ctx** out);
/* Free a context (NULL is accepted). */
int c3c_ctx_destroy(c3c_ctx* ctx);
/* Replace / read the mode bits.  EINVAL on NULL or unknown bits. */
int c3c_set_mode(c3c_ctx* ctx, uint32_t mode);
int c3c_get_mode(const c3c_ctx* ctx, uint32_t* mode);

/* ---------------------------------------------------------------- host maths */
/* Output sizes (Eq. 3 and its spatial analogue) and the new cache length
 * L = min(pad_t_base, Tc + T).  Pure host code.  Any output pointer may be
 * NULL.  EINVAL for an invalid descriptor (including Ho < 1 or Wo < 1). */
int c3c_output_dims(const c3c_conv_desc* d, int64_t* To, int64_t* Ho,
                    int64_t* Wo, int64_t* L);
/* Eq. 4: output frames [o_l, o_h) that temporal tap k contributes to
 * (source frames o + delta_k, delta_k = k dil_t - p_l).  Unit temporal stride
 * only (EINVAL otherwise); o_l >= o_h means the tap is inactive. */
int c3c_tap_interval(const c3c_conv_desc* d, int64_t k, int64_t* o_l,
                     int64_t* o_h);
/* Algorithmic FLOP of one call: 2 N Co (Ci/groups) Kh Kw Ho Wo times the
 * number of (output frame, temporal tap) pairs whose source frame lies in Z.
 * Pure host code.  EINVAL for an invalid descriptor. */
int c3c_flops(const c3c_conv_desc* d, double* flops);
/* The route the call would take under ctx's mode, with the reason.  Pure
 * host code: no device access, counters untouched.  ctx may be NULL (mode 0). */
int c3c_route_query(const c3c_ctx* ctx, const c3c_conv_desc* d, int* route,
                    int* reason);

/* ---------------------------------------------------------------- launch plan */
/* The kernels of the library.  The fast route's 3x3 form runs on
 * CONV3D_BF16 (or FAST_F32), with HEAD for few output channels; its 1x1 form
 * on TAP1X1 or POINTWISE; the fallback on POINTWISE (1x1x1 calls) or
 * FALLBACK_DIRECT. */
typedef enum c3c_kernel {
  C3C_KERNEL_NONE = 0,            /* nothing to compute (no output frame)      */
  C3C_KERNEL_CONV3D_BF16 = 1,     /* the implicit-GEMM kernel, bf16, 3x3       */
  C3C_KERNEL_HEAD = 2,            /* bf16, 3x3, Co <= 5: taps as GEMM columns  */
  C3C_KERNEL_TAP1X1 = 3,          /* bf16, 1x1: 192-channel x 128-pixel tiles  */
  C3C_KERNEL_POINTWISE = 4,       /* bf16 / f16 per-frame matrix products      */
  C3C_KERNEL_FAST_F32 = 5,        /* fp32 matrix cores, 3x3 and 1x1            */
  C3C_KERNEL_FALLBACK_DIRECT = 6  /* generic direct Conv3D, fp32 accumulation  */
} c3c_kernel;

/* What one plain call (c3c_conv3d_causal_cached) would launch: its route,
 * the main kernel and its workgroup tile, as chosen by the same code that
 * launches it.  tile_h == 0 marks a kernel that tiles the flattened Ho*Wo
 * plane: tile_w is then a run of consecutive pixels of that plane. */
typedef struct c3c_plan {
  int32_t route;           /* enum c3c_route                                 */
  int32_t reason;          /* enum c3c_reason                                */
  int32_t kernel;          /* enum c3c_kernel                                */
  int32_t splits;          /* split-K factor (1: unsplit)                    */
  int64_t tile_co;         /* output channels per workgroup                  */
  int64_t tile_h, tile_w;  /* output rows x columns per workgroup            */
  int64_t workgroups;      /* of the main launch, every split included       */
  int32_t cache_in_kernel; /* 1: the main kernel writes cache_out itself     */
  int32_t reserved;
} c3c_plan;

/* Fill *out with the plan of a plain call under ctx's mode (ctx may be NULL:
 * mode 0) with a split-K workspace of ws_bytes attached.  Pure host code; it
 * reads the current device's compute-unit count as the launch does (256 when
 * no device is visible).  The plan assumes 16-byte-aligned tensors: a call
 * with misaligned tensors may take an unaligned variant of the same tile or,
 * for HEAD and TAP1X1, the CONV3D_BF16 and POINTWISE kernels.
 * EINVAL for an invalid descriptor or NULL out. */
int c3c_plan_query(const c3c_ctx* ctx, const c3c_conv_desc* d, size_t ws_bytes,
                   c3c_plan* out);

/* ---------------------------------------------------------------- workspace */
/* Split-K workspace.  A bf16 fast call whose output tiles cannot fill the
 * device's compute units (few output frames at a low resolution, such as one
 * new frame at 60x104) can split each tile's (tap, 32-channel chunk) stages
 * -- the K dimension of the lowered GEMM, Eq. 2 summed over the active taps
 * of Eq. 4 -- over several workgroups.  Each split writes fp32 partial sums
 * to the workspace; a second kernel adds the splits in a fixed order, adds
 * the bias once and rounds once (so results are deterministic).
 *
 * c3c_workspace_bytes: the bytes a call with this descriptor would use, 0
 * when it would run unsplit (large calls, non-bf16, or not routing fast).
 * The split is planned from the compute-unit count of the device that is
 * current when the query runs (256 is assumed when no device is visible):
 * query and launch with the same device current, since a workspace sized for
 * one device can be too small for the plan on another, and the call then
 * runs unsplit.  EINVAL for an invalid descriptor or NULL bytes.
 *
 * c3c_ctx_set_workspace: attach a device buffer (caller-owned, 16-byte
 * aligned) to the context; (NULL, 0) detaches.  A call splits only when the
 * attached buffer holds at least c3c_workspace_bytes; otherwise it runs
 * unsplit, with the same results up to summation order.  The buffer must not
 * overlap any tensor of a call (EINVAL at the call), and calls that share a
 * context must not run concurrently on different streams while they use it.
 * EINVAL on NULL ctx, a NULL buffer with nonzero bytes (or the reverse), or a
 * misaligned buffer. */
int c3c_workspace_bytes(const c3c_conv_desc* d, size_t* bytes);
int c3c_ctx_set_workspace(c3c_ctx* ctx, void* ws, size_t bytes);

/* ---------------------------------------------------------------- weights */
/* Size in bytes of the packed fast-route weights for this layer (the paper's
 * derived per-tap weight slices, Alg. 1, kept as one matrix-core-ready copy).
 * 0 when the call does not route fast under mode 0. */
int c3c_weight_pack_bytes(const c3c_conv_desc* d, size_t* bytes);
/* Repack w (device, [Co][Ci][Kt][Kh][Kw]) into wpack (device, caller
 * allocated, c3c_weight_pack_bytes bytes): a bit-exact permutation into
 * K-major matrix-core fragments, zero padded to whole fragments.  Enqueued on
 * `stream`.  Re-run it whenever w changes.  EINVAL if the layer has no fast
 * layout (bytes == 0), on NULL pointers or if wpack aliases w. */
int c3c_weight_repack(c3c_ctx* ctx, const c3c_conv_desc* d, const void* w,
                      void* wpack, void* stream);
/* Inverse permutation, for tests: wpack -> w_out ([Co][Ci][Kt][Kh][Kw]). */
int c3c_weight_unpack(const c3c_conv_desc* d, const void* wpack, void* w_out,
                      void* stream);

/* ---------------------------------------------------------------- the call */
/* y = CausalConv3D([cache; x], w) + bias, cache_out = last L frames of
 * [cache; x]  (Eq. 2 with the intervals of Eq. 4; Alg. 1).
 *
 * Fast route: one kernel launch evaluates every active tap into fp32
 * registers, adds the bias once, rounds to `dtype` (nearest even), stores
 * NCTHW, and writes cache_out (3x3 kernels write it in the same launch; 1x1
 * kernels and fp32 calls copy it with a second kernel).  It reads wpack (required, from
 * c3c_weight_repack on the same w); w itself is not read.
 * Fallback route: the direct-Conv3D kernel reads w (wpack may be NULL), then a
 * copy kernel writes cache_out.
 *
 * Counters: calls++ first; then, once the call's kernels are enqueued,
 * fast++, or fallback++ with unsupported / forced / fast_error; or
 * strict_rejects++ (with C3C_E_UNSUPPORTED, C3C_E_INJECTED or C3C_E_DEVICE
 * in strict mode); or failed++ when the fallback's own launch fails
 * (C3C_E_DEVICE).  A call returning EINVAL is not counted.
 * EINVAL: NULL ctx/desc, invalid descriptor, a required pointer NULL,
 * cache_out overlapping cache or x, y overlapping any input, or wpack NULL
 * on a call that routes fast. */
int c3c_conv3d_causal_cached(c3c_ctx* ctx, const c3c_conv_desc* d,
                             const void* x, const void* cache, const void* w,
                             const void* wpack, const void* bias, void* y,
                             void* cache_out, void* stream);

/* ---------------------------------------------------------------- fused form */
/* The same call with the neighbouring ops of a decoder residual block folded
 * in (bf16 only).  Each part is optional:
 *
 *   prologue  the new chunk x is read as
 *               u = RNE_bf16(SiLU(x * scale[n][ci] + shift[n][ci])),
 *               SiLU(v) = v / (1 + e^-v), computed in fp32: a normalisation
 *             whose statistics and affine the caller has folded into one
 *             scale and shift per (batch element, input channel), then the
 *             activation.  Zero padding applies to u (padded positions stay
 *             0).  The cache holds activated frames: cache frames are read as
 *             they are, and cache_out receives the last L frames of
 *             [cache; u] -- what the cache of the convolution would hold in an
 *             unfused pipeline.
 *   epilogue  residual (y's layout and dtype) is added after the bias,
 *             before the one rounding: y = RNE(conv + bias + residual).
 *
 * The paper's memory results (Sec. 6) and discussion (Sec. 7) name the
 * temporary buffers around the lowering and point to buffer reuse and
 * streamed accumulation; this form removes the activated-input tensor and
 * the separate residual pass of an unfused block.
 *
 * scale, shift: device fp32 [N][Ci], both or neither (neither: u = x).
 * residual: device, [N][Co][To][Ho][Wo] bf16, or NULL; it may be y itself
 *   (in place) but may not otherwise overlap an output.
 * Routing, counters, strict mode and the other arguments are those of
 * c3c_conv3d_causal_cached.  With scale, shift and residual all NULL the
 * call is exactly c3c_conv3d_causal_cached.
 * EINVAL: as c3c_conv3d_causal_cached; dtype not bf16; exactly one of scale
 * and shift NULL; scale, shift or residual overlapping an output (other than
 * residual == y). */
/* Workspace for the fused form's prologue pass.  On the fast route with the
 * 3x3 spatial kernel, the prologue inside the convolution kernel evaluates
 * SiLU once per time an input element is staged (about 3.75 times: three
 * taps and the tile halo).  When the context's workspace (c3c_ctx_set_-
 * workspace) holds at least the bytes this query reports, a fused call
 * instead activates the new chunk once, in a separate elementwise pass, into
 * the workspace's first round_up(|x|, 256) bytes, and runs the convolution on
 * it (the residual stays fused; the rest of the workspace serves split-K as
 * for a plain call).  The results are identical; the pass costs |x| bytes of
 * workspace and two HBM passes over |x| instead of the repeated SiLU.
 * *bytes: that size (the prologue region plus the split-K bytes of
 * c3c_workspace_bytes), 0 when the fused call would not use a prologue pass
 * (not bf16, or not the fast 3x3 form).  EINVAL for an invalid descriptor or
 * NULL bytes. */
int c3c_fused_workspace_bytes(const c3c_conv_desc* d, size_t* bytes);

int c3c_conv3d_causal_cached_fused(c3c_ctx* ctx, const c3c_conv_desc* d,
                                   const void* x, const void* cache,
                                   const void* w, const void* wpack,
                                   const void* bias, const float* scale,
                                   const float* shift, const void* residual,
                                   void* y, void* cache_out, void* stream);

/* ---------------------------------------------------------------- normalised block form */
/* The fused form with the residual block's normalisation computed inside the
 * call instead of folded by the caller (bf16 only).  A decoder residual
 * block normalises each pixel over its channels, applies a per-channel gain
 * and bias and SiLU, then runs its cached causal convolution; the paper's
 * Sec. 7 points at the temporary buffers around the lowering (buffer reuse,
 * streamed accumulation).  Here the new chunk x becomes
 *   u[n][ci][t][p] = RNE_bf16(SiLU(x[n][ci][t][p] * r[n][t][p] * gamma[ci] + beta[ci])),
 *   r[n][t][p] = 1 / sqrt(mean over ci of x[n][ci][t][p]^2 + eps),
 * in one pass over x (fp32 arithmetic, hardware reciprocal square root,
 * exponential and reciprocal) into the first round_up(|x|, 256) bytes of the
 * context's workspace (c3c_ctx_set_workspace).  The convolution then runs on
 * [cache; u] exactly as c3c_conv3d_causal_cached does, with the rest of the
 * workspace as its split-K workspace: cache frames are read as they are,
 * cache_out receives the last L frames of [cache; u] (activated frames, as
 * the cache of an unfused pipeline would hold), and residual (or NULL) is
 * added after the bias, before the one rounding.
 *
 * gamma, beta: device fp32 [Ci].  eps: finite and >= 0.  residual: device,
 *   [N][Co][To][Ho][Wo] bf16, or NULL; it may be y itself.
 * Workspace: at least c3c_block_workspace_bytes(d) (the activated chunk,
 *   then c3c_workspace_bytes); calls sharing a context's workspace must not
 *   overlap in time.
 * EINVAL (not counted): as c3c_conv3d_causal_cached; dtype not bf16; gamma
 *   or beta NULL; eps negative, NaN or infinite; a context workspace smaller
 *   than c3c_block_workspace_bytes; x, gamma or beta overlapping an output or
 *   the workspace; residual overlapping the workspace or an output other
 *   than y.
 * Routing, counters and strict mode as c3c_conv3d_causal_cached; strict
 *   rejections happen before the pass runs; a failed pass launch counts the
 *   call as failed and returns C3C_E_DEVICE. */
int c3c_block_workspace_bytes(const c3c_conv_desc* d, size_t* bytes);
int c3c_conv3d_causal_cached_block(c3c_ctx* ctx, const c3c_conv_desc* d,
                                   const void* x, const void* cache,
                                   const void* w, const void* wpack,
                                   const void* bias, const float* gamma,
                                   const float* beta, float eps,
                                   const void* residual, void* y,
                                   void* cache_out, void* stream);

/* ---------------------------------------------------------------- no allocation */
/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the plain
 * call of c3c_conv3d_causal_cached, same arguments and results, that never
 * uses a caller workspace and allocates nothing.  A call that splits its
 * stages (split-K, see c3c_workspace_bytes) keeps its fp32 partial sums in
 * a scratch array inside the library instead: C3C_NOALLOC_SCRATCH_BYTES
 * bytes of device memory on each device the library runs on, held until the
 * process ends.  The array is looked up on the call's first use of a device
 * (no allocation).  A call whose split needs more than that returns EINVAL
 * (not counted) with a message naming both sizes.  Every call on one device
 * shares its array, which keeps the last call's partial sums: calls that
 * overlap in time on one device (several streams or host threads) race and
 * must be serialised by the caller.  The context's workspace, if any, is
 * ignored.  Routing, counters, modes and errors otherwise as for
 * c3c_conv3d_causal_cached (a failed symbol lookup is C3C_E_DEVICE, counted
 * nowhere). */
#define C3C_NOALLOC_SCRATCH_BYTES (64ll << 20)
int c3c_conv3d_causal_cached_noalloc(c3c_ctx* ctx, const c3c_conv_desc* d,
                                     const void* x, const void* cache,
                                     const void* w, const void* wpack,
                                     const void* bias, void* y,
                                     void* cache_out, void* stream);

/* ---------------------------------------------------------------- counters */
int c3c_counters_get(const c3c_ctx* ctx, c3c_counters* out);
int c3c_counters_reset(c3c_ctx* ctx); /* also clears the shape histogram */
/* Copy up to `cap` histogram entries (first-seen order) into out (host
 * memory); *n receives the total number of distinct entries. */
int c3c_fallback_shapes(const c3c_ctx* ctx, c3c_sig_count* out, int cap,
                        int* n);

/* ---------------------------------------------------------------- measurement */
/* Not part of the paper's method: a reference rate for measuring the
 * kernels.  Launches `blocks` workgroups of 4 waves; each wave runs `iters`
 * iterations of 8 independent back-to-back bf16 matrix-core products
 * (16x16x32) and reads no memory; with several workgroups per compute unit
 * the launch runs at the matrix cores' peak at the clock the device sustains
 * under that load.  Writes one float per thread to `out` (device memory,
 * blocks * 256 floats, caller-owned); *flops receives the launch's FLOP
 * count; the caller times the launch on `stream`.
 * EINVAL: blocks or iters outside [1, 2^31), out or flops NULL. */
int c3c_mfma_probe(int64_t blocks, int64_t iters, float* out, double* flops, void* stream);

/* ---------------------------------------------------------------- messages */
const char* c3c_strerror(int status);
/* Message of the last failed call on ctx ("" if none); valid until the next
 * call on ctx. */
const char* c3c_last_error(const c3c_ctx* ctx);

#ifdef __cplusplus
}
#endif
#endif /* C3C_H */
