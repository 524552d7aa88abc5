/*
 * dtst.h -- C ABI of the DTST spectral-layer library for AMD MI355X (gfx950).
 *
 * The library computes, on one GPU's shard of a spatially decomposed
 * (x, y, z, t) grid, the hot path of one Fourier-neural-operator spectral
 * layer as defined in "DRIFT: Direct Reduced Fourier Transforms for
 * Distributed Spectral Neural Operators" (arXiv 2607.14394):
 *
 *   forward partial DFT   Sec. IV-B Eq. (dtst_decompose), basis of Sec. V-B
 *                         Eq. (basis_matrix), summed over shards as in
 *                         Eq. (dtst_reduce) through the `accumulate` flag
 *   mode-wise channel mix Sec. V-A Eq. (partitioned_conv) on a mode range S_p
 *   inverse partial DFT   Sec. V-A Eq. (dtst_inverse)
 *   adjoints              Sec. V-C (backward pass)
 *
 * Conventions shared by every call
 * --------------------------------
 * Dimensions are ordered (x, y, z, t); t is innermost in memory.
 * Retained modes: x, y, z keep the stored indices {0..k-1} U {N-k..N-1}
 * (Sec. III, Fig. 5), t keeps {0..kt-1} (the half spectrum of a real
 * signal).  Within a dimension modes are stored in ascending stored index.
 * M = (2kx)(2ky)(2kz)kt and the flattened mode index is
 * m = ((ix*Ky + iy)*Kz + iz)*Kt + it.
 *
 * Basis (Sec. V-B): B_i[k, j] = exp(-2 pi i ((k * (offset_i + j)) mod N_i) / N_i);
 * the exponent is reduced in exact integer arithmetic, the trigonometric
 * value is taken in fp64 and rounded once to fp32.
 *
 * Inverse of the half spectrum: y[n] = (1/prod N) Re sum_k w(k_t) Yhat[k]
 * conj(phi_k(n)) with w(0) = 1, w(N_t/2) = 1 for even N_t, w = 2 otherwise.
 *
 * Memory: every array argument is a contiguous, row-major DEVICE pointer
 * owned by the caller, aligned to 16 bytes.  Complex arrays are interleaved
 * (re, im) fp32 pairs, the layout of torch.complex64.
 *
 *   x, y, g_x, g_y           (B, C, Nx_loc, Ny_loc, Nz_loc, Nt_loc) fp32
 *   xhat, yhat, g_xhat, ...  (B, C, 2kx, 2ky, 2kz, kt) complex64
 *   w_shard, g_w_shard       (m1 - m0, C_in, C_out) complex64
 *
 * C is C_in for forward / forward_adj / the mix input and C_out for the
 * mix output / inverse / inverse_adj.
 *
 * Execution: every execute call is asynchronous on `stream` (a hipStream_t
 * passed as void*, NULL = the default stream), allocates nothing and never
 * synchronises the host.  All validation happens on the host before any
 * launch; on an error nothing is launched, outputs are untouched and the
 * status says why (dtst_last_error() gives the detail for the calling
 * thread).  Nothing throws across the ABI and nothing aborts.  Plans are
 * immutable after creation and may be used concurrently from several
 * streams as long as each concurrent call has its own workspace.
 */
#ifndef DTST_H
#define DTST_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DTST_VERSION_MAJOR 0
#define DTST_VERSION_MINOR 1

typedef struct dtst_plan_st* dtst_plan_t; /* opaque; created and owned by the library */

typedef enum {
  DTST_OK = 0,
  DTST_ERR_INVALID_ARG = 1,   /* bad descriptor, pointer, size, range or plan */
  DTST_ERR_UNSUPPORTED = 2,   /* valid geometry outside what the kernels cover */
  DTST_ERR_OUT_OF_MEMORY = 3, /* device allocation at plan creation failed */
  DTST_ERR_DEVICE = 4         /* a HIP call or kernel launch failed */
} dtst_status;

/* Geometry of one shard (Sec. IV-A problem setting; offsets of Sec. V-B). */
typedef struct {
  int64_t n_global[4]; /* N_x, N_y, N_z, N_t of the global grid, each >= 1          */
  int64_t n_local[4];  /* local extents N_i^loc of this shard, each >= 1            */
  int64_t offset[4];   /* global index of the shard's first element, p_i N_i^loc;   */
                       /* 0 <= offset, offset + n_local <= n_global                 */
  int32_t kmax[3];     /* x, y, z keep 2k indices; need 1 <= 2k <= N (Sec. III)     */
  int32_t kt;          /* t keeps 0..kt-1; need 1 <= kt <= N_t/2 + 1                */
  int64_t batch;       /* B >= 0 (0 makes every execute call a no-op)              */
  int64_t c_in;        /* input channels  >= 1                                     */
  int64_t c_out;       /* output channels >= 1                                     */
} dtst_desc;

/* ---- host-only helpers (no GPU needed) --------------------------------- */

/* Check a descriptor.  DTST_OK, DTST_ERR_INVALID_ARG for a geometry the
 * method does not define, DTST_ERR_UNSUPPORTED for one the kernels do not
 * cover (currently: kt <= 16, N_t^loc <= 64, c_out <= 512, and per-kernel
 * LDS limits). */
dtst_status dtst_desc_validate(const dtst_desc* d);

/* Workspace bytes the execute calls of this geometry need (>= 0), for a
 * plan made with dtst_plan (the default schedule). */
dtst_status dtst_desc_workspace_bytes(const dtst_desc* d, size_t* bytes);

/* The same for a plan made with dtst_plan_ex(d, flags, ...). */
dtst_status dtst_desc_workspace_bytes_ex(const dtst_desc* d, uint32_t flags, size_t* bytes);

/* Write the fp32 basis matrix of dimension `dim` (0..3 = x, y, z, t) that
 * the plan uploads, as an interleaved complex (K_dim x N_dim^loc) host array
 * of `count` floats (count must equal 2*K_dim*N_dim^loc).  kind 0: the
 * forward basis B_dim of Eq. (basis_matrix); kind 1: conj(B_dim), the
 * inverse basis before the 1/prod N and half-spectrum weights.  Sec. V-B. */
dtst_status dtst_basis_host(const dtst_desc* d, int dim, int kind, float* out, size_t count);

/* ---- plans ------------------------------------------------------------- */

/* Validate `d`, build every basis table on the host in fp64, round to fp32
 * and upload them to the current HIP device (synchronously).  The plan is
 * bound to that device.  On success *out receives the plan.
 *
 * The plan also fixes the kernel schedule of both chains (dtst_forward and
 * dtst_inverse_adj; dtst_inverse and dtst_forward_adj): where the shapes
 * allow it (K_t <= 8, at most 16 z modes per fold class, N_t^loc <= 32 and a
 * multiple of 4, K_y <= 32, K_z K_t <= 256) the t, z and y contractions run
 * as one launch; otherwise t + z and y are separate launches.  Same as
 * dtst_plan_ex(d, 0, out). */
dtst_status dtst_plan(const dtst_desc* d, dtst_plan_t* out);

/* Plan options (bit flags of dtst_plan_ex / dtst_desc_workspace_bytes_ex). */
enum {
  /* Keep the t + z and y contractions (and the y and z + t expansions) as
   * separate launches even where the shapes allow one launch.  The result
   * agrees with the default schedule to rounding (the contraction order of
   * Sec. V-B is the same); the workspace then also holds the (.., N_x, N_y,
   * K_z, K_t) intermediate. */
  DTST_PLAN_SPLIT_SCHEDULE = 1u,
  /* Run dtst_inverse_block as the inverse followed by a separate epilogue
   * launch (the form of dtst_inverse + dtst_block_epilogue) instead of the
   * fused z + t expansion and epilogue kernel.  Same result to rounding. */
  DTST_PLAN_UNFUSED_BLOCK = 2u
};

/* dtst_plan with options: `flags` is 0 or a combination of the DTST_PLAN_*
 * flags above; any other bit is DTST_ERR_INVALID_ARG. */
dtst_status dtst_plan_ex(const dtst_desc* d, uint32_t flags, dtst_plan_t* out);

/* Free the plan's device tables.  Using a destroyed plan afterwards returns
 * DTST_ERR_INVALID_ARG. */
dtst_status dtst_plan_destroy(dtst_plan_t p);

/* Number of retained modes M and the workspace size for every execute call
 * of this plan.  Either output pointer may be NULL. */
dtst_status dtst_plan_info(dtst_plan_t p, int64_t* n_modes, size_t* workspace_bytes);

/* ---- execute calls ------------------------------------------------------ */

/* Forward partial spectrum of the shard (Sec. IV-B Eq. dtst_decompose):
 *   xhat[b,c,k] (+)= sum_{n in shard} x[b,c,n] prod_i B_i[k_i, n_i]
 * for the C_in channels.  accumulate = 0 overwrites xhat; 1 adds to it, so
 * calling it for every shard in turn forms the sum of Eq. (dtst_reduce).
 * The contraction order is t, z, y, x (Algorithm 1). */
dtst_status dtst_forward(dtst_plan_t p, const float* x, void* xhat, int accumulate,
                         void* workspace, size_t workspace_bytes, void* stream);

/* Mode-wise channel mix on the flattened mode range [m0, m1) (Sec. V-A,
 * Eq. partitioned_conv), with w_shard the local weights R_theta^(p):
 *   op 0:  yhat[b,o,m]  = sum_i xhat[b,i,m] * w[m-m0,i,o]         (xhat: C_in,  yhat: C_out)
 *   op 1:  yhat[b,i,m]  = sum_o xhat[b,o,m] * conj(w[m-m0,i,o])   (xhat: C_out, yhat: C_in)
 * op 1 is the data gradient of op 0.  Only columns m0..m1-1 of yhat are
 * written; the rest is untouched, so running the disjoint ranges one after
 * another assembles the whole spectrum.  0 <= m0 <= m1 <= M. */
dtst_status dtst_mix(dtst_plan_t p, const void* xhat, const void* w_shard, void* yhat,
                     int64_t m0, int64_t m1, int op, void* stream);

/* Inverse partial DFT onto the shard (Sec. V-A Eq. dtst_inverse, half
 * spectrum in t) for the C_out channels:
 *   y[b,c,n] = (1/prod N) Re sum_k w(k_t) yhat[b,c,k] conj(prod_i B_i[k_i, n_i]).
 * Expansion order x, y, z, t. */
dtst_status dtst_inverse(dtst_plan_t p, const void* yhat, float* y,
                         void* workspace, size_t workspace_bytes, void* stream);

/* Adjoint of dtst_forward (Sec. V-C), C_in channels:
 *   g_x[b,c,n] = Re sum_k g_xhat[b,c,k] conj(prod_i B_i[k_i, n_i]). */
dtst_status dtst_forward_adj(dtst_plan_t p, const void* g_xhat, float* g_x,
                             void* workspace, size_t workspace_bytes, void* stream);

/* Adjoint of dtst_inverse (Sec. V-C), C_out channels:
 *   g_yhat[b,c,k] (+)= (w(k_t)/prod N) sum_n g_y[b,c,n] prod_i B_i[k_i, n_i]. */
dtst_status dtst_inverse_adj(dtst_plan_t p, const float* g_y, void* g_yhat, int accumulate,
                             void* workspace, size_t workspace_bytes, void* stream);

/* Gradient of the local weights on [m0, m1) (Sec. V-A, Sec. V-C; local, no
 * synchronisation needed):
 *   g_w[m-m0,i,o] (+)= sum_b conj(xhat[b,i,m]) * g_yhat[b,o,m]. */
dtst_status dtst_mix_wgrad(dtst_plan_t p, const void* xhat, const void* g_yhat, void* g_w_shard,
                           int64_t m0, int64_t m1, int accumulate, void* stream);

/* Point-wise linear layer over the points of a (B, C, points) tensor: the
 * lift P and the projection Q that the FNO applies before and after its
 * Fourier layers (Sec. II), read as single linear layers with a bias:
 *   y[b,o,n] = act( sum_i w[o,i] x[b,i,n] + bias[o] ),
 * act = 0: identity, act = 1: GELU(v) = v (1 + erf(v / sqrt 2)) / 2.
 * x: (batch, c_in, points) fp32; y: (batch, c_out, points) fp32; w: (c_out,
 * c_in) fp32 row-major; bias: c_out fp32, or NULL for none.  Device arrays
 * owned by the caller, 16-byte aligned; x must not overlap y
 * (DTST_ERR_INVALID_ARG); c_in * c_out + c_out <= 40960 (DTST_ERR_UNSUPPORTED).
 * Independent of any plan; runs on the current device, asynchronous on
 * `stream`, no allocation. */
dtst_status dtst_pointwise(const float* x, const float* w, const float* bias, float* y, int64_t batch,
                           int64_t c_in, int64_t c_out, int64_t points, int act, void* stream);

/* Block epilogue (Sec. V block structure; Algorithm 1, first and last step):
 * the point-wise linear bypass of the block input added to the spectral
 * output, through the activation, in place on y:
 *   y[b,o,n] <- GELU( sum_i w_bypass[o,i] x[b,i,n] + y[b,o,n] ),
 *   GELU(v) = v Phi(v) = v (1 + erf(v / sqrt 2)) / 2  (exact form, no bias).
 * x: (B, C_in, shard) fp32, the block input; y: (B, C_out, shard) fp32, the
 * output of dtst_inverse; w_bypass: (C_out, C_in) fp32 row-major.  All are
 * device arrays owned by the caller, 16-byte aligned; x must not overlap y
 * (DTST_ERR_INVALID_ARG); C_in * C_out <= 40960 (DTST_ERR_UNSUPPORTED).
 * Asynchronous on `stream`, no allocation. */
dtst_status dtst_block_epilogue(dtst_plan_t p, const float* x, const float* w_bypass, float* y, void* stream);

/* The block's last step in one call (Algorithm 1, last step; Eq.
 * dtst_inverse for the spectral part): the inverse partial DFT of yhat
 * followed by the block epilogue,
 *   y = GELU( w_bypass x + inverse(yhat) ),
 * with the arrays, layouts, alignment and overlap rules of dtst_inverse and
 * dtst_block_epilogue.  Where the plan allows it (N_t^loc a multiple of 4 and
 * at most 32, C_in and C_out at most 32, at most 32 z modes per fold class,
 * the per-workgroup buffers within the LDS; see
 * dtst_plan_block_workspace_bytes) the z and t expansions and the epilogue
 * run as one kernel that writes y once and reads x once; otherwise, or with
 * DTST_PLAN_UNFUSED_BLOCK, the inverse and the epilogue are enqueued one
 * after the other.  The workspace must hold
 * dtst_plan_block_workspace_bytes(p) bytes (DTST_ERR_INVALID_ARG otherwise);
 * it is scratch, owned by the caller.  Asynchronous on `stream`, no
 * allocation. */
dtst_status dtst_inverse_block(dtst_plan_t p, const void* yhat, const float* x, const float* w_bypass, float* y,
                               void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes dtst_inverse_block needs with this plan (at least the
 * workspace of dtst_plan_info; larger where the layer's own calls fuse the y
 * expansion and the block kernel reads the y-expanded (B, C_out, N_x, N_y,
 * K_z, K_t) intermediate), and whether it runs the fused kernel (1) or the
 * two launches (0).  Either output may be null. */
dtst_status dtst_plan_block_info(dtst_plan_t p, size_t* workspace_bytes, int* fused);

/* ---- no-allocation variant ------------------------------------------------ */

/* For callers that cannot allocate device memory or hand over a workspace:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same computation, arguments and errors as dtst_forward, with
 * the library's own per-device scratch array of DTST_SCRATCH_BYTES as the
 * workspace, so the call allocates nothing (no hipMalloc, no allocating
 * library routine).  Every GPU the library runs on holds its own array from
 * the time the library is loaded until the process ends.  A plan whose
 * workspace (dtst_plan_info) exceeds DTST_SCRATCH_BYTES gets
 * DTST_ERR_UNSUPPORTED and nothing is launched.  Every call on one GPU
 * shares that GPU's array and the array keeps the last call's contents:
 * calls that overlap in time on one GPU (other streams, threads or plans)
 * race and give undefined results, so the caller serialises them.  Nothing
 * in the array needs clearing: a call reads only entries it wrote before. */
#define DTST_SCRATCH_BYTES ((size_t)64 << 20)
dtst_status dtst_forward_noalloc(dtst_plan_t p, const float* x, void* xhat, int accumulate, void* stream);

/* ---- instrumentation ----------------------------------------------------- */

/* Per-kernel device time, for callers that time the path (benchmarks,
 * tuning).  While enabled, every kernel the execute calls launch is
 * bracketed by a pair of HIP events recorded on the call's stream; nothing
 * else changes.  Process-wide; off by default. */
typedef struct {
  char name[40];     /* kernel role, e.g. "stream_fwd_tzy", "stream_fwd_tz", "axis_fwd_y", "mix" */
  int64_t launches;  /* launches collected */
  double total_ms;   /* summed event-to-event device time */
} dtst_kernel_time;

dtst_status dtst_profile_enable(int on);

/* Wait for every recorded launch, write up to `capacity` per-kernel totals
 * (only kernels with launches > 0) to `out`, set *count, and reset the
 * totals.  Synchronises the host with the recorded events. */
dtst_status dtst_profile_collect(dtst_kernel_time* out, int capacity, int* count);

/* ---- diagnostics -------------------------------------------------------- */
const char* dtst_status_string(dtst_status s);
/* Detail of the last error on the calling thread ("" if none). */
const char* dtst_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DTST_H */
