/*
 * littlebit.h -- C ABI of the MI355X (gfx950) LittleBit linear-layer library.
 *
 * A LittleBit linear layer (arXiv 2506.13771, Sec. 3.1 and Sec. 3.3) replaces
 * a dense weight W in R^{d_out x d_in} by two paths p in {primary, residual},
 * each made of two sign matrices U_p in {-1,+1}^{d_out x r},
 * V_p in {-1,+1}^{d_in x r} and three scale vectors h_p in R^{d_out},
 * g_p in R^{d_in}, l_p in R^r.  The effective weight
 *     W_hat = sum_p diag(h_p) U_p diag(l_p) V_p^T diag(g_p)
 * (Eqs. w_primary_hat, res_approx_structure, final_weight_approx_res) is never
 * formed on the forward path; Proposition 1 (Eq. proposition1) evaluates
 *     y = sum_p h_p (.) ( U_p ( l_p (.) ( V_p^T ( g_p (.) x ) ) ) )
 * as two binary contractions plus element-wise scalings.
 *
 * Conventions for every call:
 *   - Buffer pointers are DEVICE pointers owned by the caller unless the
 *     comment says "host".  The library allocates nothing and keeps no state
 *     between calls; all state lives in caller-provided buffers.
 *   - GPU calls are asynchronous on `stream` (0 = the null stream).  Results
 *     are valid once the stream has been synchronised.
 *   - Every argument is validated on the host before anything is enqueued; a
 *     failed validation returns its code and enqueues nothing.  After a launch,
 *     a launch error reported by the HIP runtime is returned as LB_ERR_HIP.
 *     No call aborts, prints or throws across this boundary.
 *   - Shapes are int64; every dimension may be any value >= 0 (ragged sizes
 *     are supported by all kernels).  Products that index a buffer must stay
 *     below 2^31 elements (LB_ERR_SHAPE otherwise).
 *   - Dense activation and scale buffers are contiguous row-major, aligned to
 *     their element size (LB_ERR_ALIGN otherwise).  Packed sign buffers are
 *     4-byte aligned.  Workspaces are 256-byte aligned.
 *
 * Packed sign layout "LB layout v1" (the paper only states that signs are
 * packed into uint32 words, Appendix "Inference Efficiency Analysis"):
 *   A sign matrix is seen as M[o][q] with o the output index and q the
 *   reduction index of the stage that reads it:
 *     LB_ROLE_U: M = U_sign   (o = i < d_out, q = k < r),    rows = d_out
 *     LB_ROLE_V: M = V_sign^T (o = k < r,     q = j < d_in), rows = d_in
 *   bit(o,q) = 1 iff the source value is < 0 (sign -1); sign(+0) = sign(-0)
 *   = +1.  With nb = n_red / 32 and w = n_red - 32 nb:
 *     region A: uint32 A[nb][n_out], output index fastest; bit t (LSB = 0)
 *               of A[b][o] is bit(o, 32 b + t);
 *     region B: absent if w == 0; uint16 B[n_out] if 1 <= w <= 16; uint32
 *               B[n_out] if 17 <= w <= 31; bit t of B[o] is bit(o, 32 nb + t)
 *               for t < w and 0 above (pad bits are zero).
 *   Region B starts at byte 4 nb n_out; words are little-endian.
 */
#ifndef LITTLEBIT_H
#define LITTLEBIT_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LB_ABI_VERSION 7

typedef enum lb_status {
  LB_OK = 0,
  LB_ERR_NULL = 1,      /* a required pointer is NULL                              */
  LB_ERR_SHAPE = 2,     /* negative dimension, or a size beyond the 2^31 limit      */
  LB_ERR_DTYPE = 3,     /* dtype code not accepted by this call                     */
  LB_ERR_ALIGN = 4,     /* pointer not aligned as the conventions above require     */
  LB_ERR_WORKSPACE = 5, /* workspace smaller than lb_forward_workspace_bytes()      */
  LB_ERR_HIP = 6,       /* the HIP runtime reported an error for a launch           */
  LB_ERR_ARG = 7        /* any other invalid argument (enum value out of range ...) */
} lb_status;

typedef enum lb_dtype { LB_F32 = 0, LB_F16 = 1, LB_BF16 = 2 } lb_dtype;

typedef enum lb_role { LB_ROLE_U = 0, LB_ROLE_V = 1 } lb_role;

/* Which forward kernel lb_linear_forward_kernel() runs. */
typedef enum lb_kernel {
  LB_KERNEL_AUTO = 0,         /* DECODE for T <= 2; from T = 3 DECODE_MFMA while T r d_out is
                                 small (T < 16, or T < 32 with r d_out < 3e6, and r d_out < 8e6),
                                 PREFILL otherwise (each where its size limits allow) */
  LB_KERNEL_DECODE = 1,       /* single launch, 4-bit look-up tables, fp32 sign-flip accumulation;
                                 T <= 4, r <= 1024 */
  LB_KERNEL_PREFILL = 2,      /* three launches of matrix-core (MFMA) tiles with exact bf16 term
                                 products (latent sums, latent scale and term split, outputs);
                                 any size within 32-bit buffer offsets */
  LB_KERNEL_DECODE_MFMA = 3   /* single launch, matrix-core contractions: stage 1 multiplies exact
                                 bf16 terms of x by the signs carried on exact bf16 terms of g,
                                 stage 2 the +-1 signs of U by bf16 terms of l (.) z; T <= 64,
                                 r <= 832 */
} lb_kernel;

/* One path's parameters (Sec. 3.1 Eq. ghl_scales_combined; Sec. 3.3).
   U: packed U_sign, LB_ROLE_U, lb_packed_bytes(LB_ROLE_U, d_out, r) bytes.
   V: packed V_sign, LB_ROLE_V, lb_packed_bytes(LB_ROLE_V, d_in, r) bytes.
   h [d_out], g [d_in], l [r]: scales in the call's scale dtype.
   A layer without the residual path is expressed by a residual path whose
   h is all zeros (the bits-per-weight note under Eq. b_calculation). */
typedef struct lb_path {
  const void* U;
  const void* V;
  const void* h;
  const void* g;
  const void* l;
} lb_path;

/* ABI version of the loaded library (LB_ABI_VERSION). */
int lb_abi_version(void);

/* Static, NUL-terminated name of a status code. */
const char* lb_status_str(lb_status s);

/* Host, pure.  Bytes of one packed sign matrix in LB layout v1; rows = d_out
   for LB_ROLE_U and d_in for LB_ROLE_V.  Returns 0 for invalid arguments. */
size_t lb_packed_bytes(lb_role role, int64_t rows, int64_t r);

/* Host, pure.  Bits per weight of a layer with `npaths` (1 or 2) paths of rank
   r (Appendix "Average Bits Per Weight Calculation", Eq. b_calculation: one
   bit per sign element, 16 bits per scale element).  Returns -1 for invalid
   arguments. */
double lb_bits_per_weight(int64_t d_in, int64_t d_out, int64_t r, int npaths);

/* Host, pure.  Per-path rank for a target bits-per-weight `bpw` with both
   paths: the largest multiple of `mult` (>= 1) whose total bits stay within
   bpw * d_in * d_out (Eq. b_calculation solved for r, Eq. r_calculation,
   rounded down to a multiple of mult).  Returns -1 for invalid arguments. */
int64_t lb_rank_for_bpw(int64_t d_in, int64_t d_out, double bpw, int64_t mult);

/* Pack the signs of a real matrix src [rows x r] (row-major, src_dtype F32,
   F16 or BF16; the latent factor U [d_out x r] for LB_ROLE_U or V [d_in x r]
   for LB_ROLE_V) into dst (lb_packed_bytes(role, rows, r) bytes) following
   Sec. 3.1 Eq. uv_sign and LB layout v1.  NaN elements are written as +1 and
   counted: if nan_count (a device int32) is not NULL, the number of NaNs met
   is atomically added to it.  dst must not overlap src. */
lb_status lb_pack_signs(const void* src, lb_dtype src_dtype, int64_t rows, int64_t r, lb_role role,
                        void* dst, int32_t* nan_count, hipStream_t stream);

/* Host, pure.  Workspace bytes lb_linear_forward() needs for these sizes
   (covers every kernel choice).  The workspace must be zero-filled once before
   its first use (lb_workspace_init does it); every call leaves it ready for
   the next one, so a workspace is reused without clearing, across calls of
   any shape.  The decode kernel tags its intermediate values with a 32-bit
   call counter kept in the workspace; a value left unread for exactly 2^32
   calls could be mistaken for a fresh one.  Calls that may run concurrently
   need distinct workspaces. */
size_t lb_forward_workspace_bytes(int64_t T, int64_t d_in, int64_t d_out, int64_t r);

/* Zero-fill a workspace of `bytes` bytes on `stream`. */
lb_status lb_workspace_init(void* workspace, size_t bytes, hipStream_t stream);

/* Read and clear the error word of a workspace used by lb_linear_forward,
   lb_linear_forward_kernel or lb_linear_forward_many (the word sits in the
   control block at the start of the workspace; one word per workspace, shared
   by every call that used it).  Enqueued on `stream`: *status (a DEVICE int32,
   4-byte aligned) receives the word and the word is reset to 0.  0 means no
   bounded wait of the single-launch decode kernels expired since the last
   clear.  Nonzero (bit 0) means one did: a workgroup gave up waiting for
   partial sums of another workgroup of the same call, took the values it
   never saw as NaN (so the affected outputs are NaN, never stale values of an
   earlier call) and set the word; the outputs of the calls since the last
   clear are then not to be trusted.  Bit 1: lb_list_forward found a plan that
   does not match its descriptors and computed nothing.  workspace_bytes must
   be at least the 256 bytes of the control block (LB_ERR_WORKSPACE).  For a
   workspace of lb_list_* the word is part of the plan's header. */
lb_status lb_workspace_status(void* workspace, size_t workspace_bytes, int32_t* status, hipStream_t stream);

/* Largest token count LB_KERNEL_DECODE accepts. */
int64_t lb_decode_max_tokens(void);

/* Forward of one LittleBit linear layer with both paths (Proposition 1,
   Eq. proposition1, summed over the two paths, Eq. final_weight_approx_res):
     y[t][i] = sum_p h_p[i] sum_k U_p[i][k] l_p[k] sum_j V_p[j][k] g_p[j] x[t][j]
   x [T x d_in] in act_dtype (F32, F16 or BF16); y [T x d_out] in act_dtype,
   rounded once (round-to-nearest-even) from the fp32 sum of both paths;
   paths[0] = primary, paths[1] = residual, scales in scale_dtype (F32, F16 or
   BF16).  Accumulation is fp32.  The look-up-table decode kernel uses exact
   fp32 products; the matrix-core kernels multiply exact bf16 terms (the
   stored x and g cut into 1, 2 or 3 terms, the V sign carried on the g
   terms; then the +-1 U signs times l (.) z cut into two bf16 terms, 16
   significant bits, for bf16/f16 outputs, or three, the full fp32
   significand, for fp32 outputs).  If d_in == 0 or r == 0, y is zero-filled.
   workspace: >= lb_forward_workspace_bytes(T, d_in, d_out, r) bytes. */
lb_status lb_linear_forward(const void* x, lb_dtype act_dtype, int64_t T, int64_t d_in, int64_t d_out,
                            int64_t r, const lb_path* paths, lb_dtype scale_dtype, void* y,
                            void* workspace, size_t workspace_bytes, hipStream_t stream);

/* For callers that cannot allocate (code under HIP graph capture, tight
   serving loops, harnesses that forbid allocation): lb_linear_forward with no
   workspace argument.  The workspace is a static scratch array of the library,
   lb_noalloc_scratch_bytes() = 32 MiB per GPU, one copy per device, held until
   the process ends; the call allocates nothing (no hipMalloc, no allocating
   library routine).  Sizes whose lb_forward_workspace_bytes exceed the
   scratch return LB_ERR_WORKSPACE; other checks and results as for
   lb_linear_forward (bit-identical to it).  The first call on a device
   resolves that device's copy and enqueues its zero fill on `stream`; that
   first call must not be captured in a graph (LB_ERR_ARG), later ones may be.
   Every call on one GPU shares its scratch (the decode kernels keep their
   call counter there, so consecutive calls on one device need no clearing):
   calls that may overlap on one GPU (other streams, other host threads)
   race and must not be issued. */
size_t lb_noalloc_scratch_bytes(void);
lb_status lb_linear_forward_noalloc(const void* x, lb_dtype act_dtype, int64_t T, int64_t d_in, int64_t d_out,
                                    int64_t r, const lb_path* paths, lb_dtype scale_dtype, void* y,
                                    hipStream_t stream);

/* lb_linear_forward with an explicit kernel choice (any kernel accepts any
   valid input; AUTO is what lb_linear_forward uses). */
lb_status lb_linear_forward_kernel(const void* x, lb_dtype act_dtype, int64_t T, int64_t d_in,
                                   int64_t d_out, int64_t r, const lb_path* paths, lb_dtype scale_dtype,
                                   void* y, void* workspace, size_t workspace_bytes, lb_kernel kernel,
                                   hipStream_t stream);

/* One linear of a list for lb_linear_forward_many: the arguments
   lb_linear_forward takes for it. */
typedef struct lb_linear_desc {
  const void* x;
  lb_dtype act_dtype;
  int64_t T, d_in, d_out, r;
  lb_path paths[2];
  lb_dtype scale_dtype;
  void* y;
} lb_linear_desc;

/* Host, pure.  Workspace bytes lb_linear_forward_many needs for this list: a
   4352-byte list header (the control block of the decode kernels' call
   protocol, shared by every linear, and 16 counter lines of the linears of a
   list launch) plus the sum of lb_forward_workspace_bytes of its linears, each
   rounded up to 256 bytes (0 if n <= 0, descs is NULL or a size is invalid).
   Linear i uses the slice after the header and those of linears 0 .. i-1 for
   its intermediate values.  The zero-fill-once and reuse rules of
   lb_forward_workspace_bytes hold for the whole workspace, across lists of any
   layout and single calls on the same buffer (the call tags live in the
   shared control block, so they never repeat). */
size_t lb_forward_many_workspace_bytes(const lb_linear_desc* descs, int64_t n);

/* Forward of n independent LittleBit linears (each as lb_linear_forward
   computes it, Proposition 1 summed over both paths; the paper's end-to-end
   decoding measurement replaces every nn.Linear of the model by this
   forward, appendix "End-to-End Decoding Throughput"), enqueued on one
   stream with fewer launches: consecutive linears for which the automatic
   choice is the same decode kernel (look-up-table or matrix-core) and that
   share the activation and scale dtypes run as one launch of that kernel per
   up to 16 linears; every other linear (prefill sizes) is its own call with
   the automatic kernel choice.  Results are those of lb_linear_forward for each
   linear.  descs: host array of n descriptors (device pointers inside, as
   for lb_linear_forward).  No y may overlap another linear's x or y (they run
   concurrently): LB_ERR_ARG.  Every descriptor is validated as
   lb_linear_forward validates its arguments, and the whole list before
   anything is enqueued; n == 0 enqueues nothing.  workspace: 256-byte
   aligned, >= lb_forward_many_workspace_bytes(descs, n) bytes. */
lb_status lb_linear_forward_many(const lb_linear_desc* descs, int64_t n, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream);

/* Streaming list forward of decode-sized linears: the decoding step of a
   model in which every nn.Linear is a LittleBit linear (appendix "End-to-End
   Decoding Throughput"), e.g. all linears of all layers of a model for a
   batch of independent inputs, or the q/k/v or gate/up projections of one
   layer.  Each linear is computed as lb_linear_forward computes it
   (Proposition 1, Eq. proposition1, both paths, Eq. final_weight_approx_res);
   the whole list takes three kinds of launch (latent partial sums of every
   linear, their sums times l, every output), with no workgroup waiting for
   another.
     - Lists whose linears all have 1 <= T <= 2 tokens run on the look-up-
       table kernels: each result is bit-identical to
       lb_linear_forward_kernel(..., LB_KERNEL_DECODE) for that linear.
     - Lists with a linear of 3 <= T <= 64 tokens run on the matrix-core
       kernels (every linear of the list): g and x enter as exact bf16 terms,
       products are exact and sums fp32, w enters stage 2 as 2 bf16 terms
       (3 for fp32 activations); results meet the tolerance of
       lb_linear_forward, and repeated calls give the same bits.

   Scope: every linear with work has r <= 1024 and the list shares one
   activation and one scale dtype; for the look-up-table kernels a d_in whose
   runs fit them (d_in <= 32768 at r <= 1024 is always accepted); for the
   matrix-core kernels T <= 64, d_in a multiple of 4 and x, g_0, g_1 aligned
   to four elements (LB_ERR_SHAPE / LB_ERR_DTYPE otherwise); linears with
   T == 0 or d_out == 0 are skipped, those with d_in == 0 or r == 0 get
   y = 0.  n <= 65535.  No y may overlap another linear's x or y (LB_ERR_ARG);
   other checks as for lb_linear_forward.

   The list's descriptors live in the workspace (the "plan"):
   lb_list_workspace_bytes: host, pure; bytes of a workspace for this list
     (0 if the list is invalid or out of scope).
   lb_list_init: writes the plan for descs into workspace (256-byte aligned,
     >= lb_list_workspace_bytes bytes) and waits for the copy on `stream`
     (it synchronises the stream, so it cannot be captured in a graph); call
     it again whenever any field of any descriptor changes (pointers
     included).
   lb_list_forward: the forward of the list whose plan is in workspace;
     asynchronous and capturable.  descs must be the array lb_list_init saw
     (same values): the kernels compare a fingerprint of descs with the plan's
     and, if they differ, write nothing but bit 1 of the workspace's error
     word (lb_workspace_status). */
size_t lb_list_workspace_bytes(const lb_linear_desc* descs, int64_t n);
lb_status lb_list_init(const lb_linear_desc* descs, int64_t n, void* workspace, size_t workspace_bytes,
                       hipStream_t stream);
lb_status lb_list_forward(const lb_linear_desc* descs, int64_t n, void* workspace, size_t workspace_bytes,
                          hipStream_t stream);

/* Latent K/V cache (paragraph "KV Cache Compression", Fig. kv_cache_viz,
   Table kv_cache_reduction: applied to the key and value projections, the
   factored forward lets a cache hold rank-r vectors per token instead of
   d_model-wide ones).  The cached vector of token t and path p is the scaled
   stage-1 latent of Proposition 1,
     w[t][p][k] = l_p[k] sum_j V_p[j][k] g_p[j] x[t][j],
   stored token-major: w [T x 2 x r] in latent_dtype (F32, F16 or BF16),
   element (t, p, k) at (2 t + p) r + k, so that the latents of new tokens are
   appended to a cache as one contiguous run.  16-bit latents are rounded to
   nearest even from fp32.  For T >= 5 an F32 cache holds the fp32 values the
   prefill kernels compute, and lb_linear_from_latent on it gives bit for bit
   what lb_linear_forward_kernel(..., LB_KERNEL_PREFILL) gives for the same x.

   lb_linear_latent: w of x [T x d_in] (act_dtype).  Only V, g and l of the
   paths are read (U and h may be NULL).  T <= 4 (a decoding step): one launch
   that forms g (.) x in fp32 and adds it with the signs of V in fp32; larger
   T: stage 1 of the prefill kernels (exact bf16 term products, fp32
   accumulation), then one pass that sums its partial results, scales by l and
   stores w.  d_in == 0 zero-fills w.  w must not overlap x (LB_ERR_ARG).
   workspace: 256-byte aligned, >= lb_latent_workspace_bytes(T, d_in, r) bytes
   (no zero-fill needed). */
size_t lb_latent_workspace_bytes(int64_t T, int64_t d_in, int64_t r);
lb_status lb_linear_latent(const void* x, lb_dtype act_dtype, int64_t T, int64_t d_in, int64_t r,
                           const lb_path* paths, lb_dtype scale_dtype, void* w, lb_dtype latent_dtype,
                           void* workspace, size_t workspace_bytes, hipStream_t stream);

/* lb_linear_from_latent: the output of the layer from cached latents,
     y[t][i] = sum_p h_p[i] sum_k U_p[i][k] w[t][p][k],
   w [T x 2 x r] (latent_dtype) as lb_linear_latent writes it, y [T x d_out]
   in out_dtype (F32, F16 or BF16), rounded once from the fp32 sum of both
   paths.  Only U and h of the paths are read (V, g and l may be NULL).  One
   pass cuts w into bf16 terms (two for 16-bit outputs, three for fp32 ones,
   as lb_linear_forward does), then stage 2 of the prefill kernels.  r == 0
   zero-fills y.  y must not overlap w (LB_ERR_ARG).  workspace: 256-byte
   aligned, >= lb_from_latent_workspace_bytes(T, r) bytes (no zero-fill
   needed). */
size_t lb_from_latent_workspace_bytes(int64_t T, int64_t r);
lb_status lb_linear_from_latent(const void* w, lb_dtype latent_dtype, int64_t T, int64_t d_out, int64_t r,
                                const lb_path* paths, lb_dtype scale_dtype, void* y, lb_dtype out_dtype,
                                void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Training-time inputs and gradient outputs of one path for
   lb_linear_backward.  All float arrays are fp32, row-major, 4-byte aligned,
   owned by the caller; gradients are written, not accumulated, and no
   gradient array may overlap an input or another output (not checked). */
typedef struct lb_path_train {
  const float* U_latent;  /* [d_out x r] real latent factor whose signs are U_p */
  const float* V_latent;  /* [d_in x r] real latent factor whose signs are V_p */
  const void* Ut;         /* U_p's signs packed with LB_ROLE_V (rows = d_out):
                             lb_pack_signs(U_latent, LB_F32, d_out, r, LB_ROLE_V, ...) */
  const void* Vt;         /* V_p's signs packed with LB_ROLE_U (rows = d_in):
                             lb_pack_signs(V_latent, LB_F32, d_in, r, LB_ROLE_U, ...) */
  float* dU;              /* out [d_out x r]: dL/dU_latent */
  float* dV;              /* out [d_in x r]:  dL/dV_latent */
  float* dh;              /* out [d_out] */
  float* dg;              /* out [d_in] */
  float* dl;              /* out [r] */
} lb_path_train;

/* Host, pure.  Workspace bytes lb_linear_backward needs (0 for invalid sizes);
   no zero-fill needed. */
size_t lb_backward_workspace_bytes(int64_t T, int64_t d_in, int64_t d_out, int64_t r);

/* Backward of one LittleBit linear for quantization-aware training (Sec. 4
   "Training Details"; Appendix "SmoothSign versus Straight-Through
   Estimator").  Given x [T x d_in] and the upstream gradient dy = dL/dy
   [T x d_out] (both act_dtype), the chain rule through Proposition 1 for both
   paths, with a = g (.) x, z = a V, w = l (.) z, dw = (h (.) dy) U, dz = l (.) dw:
     dx      = sum_p g_p (.) (dz_p V_p^T)                (act_dtype, one rounding;
                                                          skipped if dx is NULL)
     dh_p    = rowsum(U_p (.) (dy^T w_p)),   dg_p = rowsum(V_p (.) (x^T dz_p))
     dl_p    = sum_t dw_p (.) z_p
     dU_p    = h_p (.) (dy^T w_p) (.) s'(U_latent),  dV_p = g_p (.) (x^T dz_p) (.) s'(V_latent)
   where the signs U_p, V_p are those of the latent factors (a value < 0 is
   -1) and s'(u) = kappa sech^2(kappa u), the derivative of tanh(kappa u) that
   SmoothSign uses in place of the sign's (the paper uses kappa = 100).
   paths: V (packed with LB_ROLE_V, as for the forward), h, g and l are read;
   U may be NULL.  train[2]: the latent factors, their signs packed in the
   other orientation, and the gradient outputs.  The binary contractions run
   on the prefill kernels (exact bf16 term products, fp32 accumulation); the
   two contractions over tokens run on the matrix cores with exact bf16 terms
   (three for w and dz) and fp32 accumulation.  Any size may be 0 (the
   non-empty gradients are then zero).  dx must not overlap x or dy
   (LB_ERR_ARG).  kappa must be finite and > 0 (LB_ERR_ARG).  workspace:
   256-byte aligned, >= lb_backward_workspace_bytes(T, d_in, d_out, r). */
lb_status lb_linear_backward(const void* x, const void* dy, lb_dtype act_dtype, int64_t T, int64_t d_in,
                             int64_t d_out, int64_t r, const lb_path* paths, lb_dtype scale_dtype,
                             const lb_path_train* train, float kappa, void* dx, void* workspace,
                             size_t workspace_bytes, hipStream_t stream);

/* ---- Dual-SVID conversion of a dense weight ------------------------------ */

/* Outputs of one path of lb_dual_svid (device, fp32, row-major, caller-owned):
   the latent factors whose signs are the path's sign matrices (pack them with
   lb_pack_signs: U_latent with LB_ROLE_U, V_latent with LB_ROLE_V) and the
   scales. */
typedef struct lb_svid_out {
  float* U_latent; /* [d_out x r]: U' = U_r diag(sqrt(sigma)), signed */
  float* V_latent; /* [d_in x r]:  V' = V_r diag(sqrt(sigma)) */
  float* h;        /* [d_out]: h0 */
  float* g;        /* [d_in]:  g0 */
  float* l;        /* [r]:     l0 = l_u (.) l_v */
  float* sigma;    /* [r] or NULL: the path's top r singular values, descending */
} lb_svid_out;

/* Host, pure.  Workspace bytes lb_dual_svid needs (0 if the sizes are not
   accepted): 8 * d_out * d_in bytes for the residual weight plus
   O((d_out + d_in) * (r + oversample) + 64 (r + oversample)^2) doubles. */
size_t lb_dual_svid_workspace_bytes(int64_t d_out, int64_t d_in, int64_t r, int64_t oversample);

/* Dual-SVID initialisation of a LittleBit linear from a dense weight W
   [d_out x d_in] (row-major, device, w_dtype f32 / f16 / bf16) at rank r
   (Sec. 3.2 "Dual-SVID Initialization", Eqs. sign_init_concise,
   scale_init_rank1_concise, latent_scale_init_concise_0; Sec. 3.3 "Residual
   Compensation").  Path 0 from W, path 1 from W_res = W - W_hat_pri,0 with
   W_hat_pri,0 = diag(h0) sign(U') diag(l0) sign(V')^T diag(g0).  Per path:
     - the top-r singular triplets of the path's weight, by block subspace
       iteration in fp64 (block b = min(r + oversample, d_out, d_in), `iters`
       rounds of multiplication by W^T and W, each followed by
       orthonormalisation, then a Rayleigh-Ritz step), the start block drawn
       from SplitMix64 at `seed`; the error of singular pair k decays like
       (sigma_{b+1} / sigma_k)^(2 iters + 1);
     - each pair signed so that the left vector's entry of largest magnitude
       is positive (the first on a tie); U' and V' split each singular value
       evenly;
     - h0, l_u from the best rank-1 approximation of |U'| and g0, l_v from
       that of |V'| (top singular value split evenly, signed so that h0 and g0
       sum to >= 0); l0 = l_u (.) l_v.
   sign() is -1 iff a value is < 0.  Outputs per path in out[0], out[1] (host
   array of two; every pointer but sigma required, fp32, 4-byte aligned);
   W_res [d_out x d_in] fp32 is written when not NULL.  Sizes: 1 <= r <=
   min(d_out, d_in), oversample >= 0, min(r + oversample, d_out, d_in) <= 1024,
   0 <= iters <= 1000 (LB_ERR_SHAPE / LB_ERR_ARG otherwise).  workspace:
   256-byte aligned, lb_dual_svid_workspace_bytes bytes, no zero-fill needed.
   Deterministic: the same inputs and seed give the same bits. */
lb_status lb_dual_svid(const void* W, lb_dtype w_dtype, int64_t d_out, int64_t d_in, int64_t r, int64_t oversample,
                       int32_t iters, uint64_t seed, const lb_svid_out* out, float* W_res, void* workspace,
                       size_t workspace_bytes, hipStream_t stream);

/* Checking path: the dense effective weight of both paths,
     W[i][j] = sum_p h_p[i] g_p[j] sum_k U_p[i][k] l_p[k] V_p[j][k]
   (Eqs. w_primary_hat, res_approx_structure, final_weight_approx_res),
   computed from the PACKED buffers in fp32 (ascending k), written to
   W [d_out x d_in] row-major fp32.  Not used by the forward path. */
lb_status lb_dense_reference_weight(const lb_path* paths, lb_dtype scale_dtype, int64_t d_in,
                                    int64_t d_out, int64_t r, float* W, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* LITTLEBIT_H */
