/*
 * graphleap.h -- C ABI of the MI355X (gfx950) GraphLeap graph-convolution path.
 *
 * The operations follow the paper "GraphLeap: Decoupling Graph Construction
 * and Convolution for Vision GNN Acceleration on FPGA":
 *   - the dynamic kNN image graph G(X) of Sec. II-B (Eq. 4), built as in the
 *     Graph Construction Engine of Sec. IV-B (pairwise distances of Alg. 2,
 *     per-node selection of the k nearest, dilation);
 *   - max-relative graph convolution MRConv of Sec. II-A (Eq. 2 and Eq. 3),
 *     with the weight split W_x / W_m of Sec. IV-C2;
 *   - the GraphLeap lookahead of Sec. III (Eq. 10-12, Alg. 1): block l's
 *     update uses the graph built from block l-1's features while the graph
 *     for block l+1 is built concurrently (Sec. IV-A, IV-F).
 *
 * Conventions for every call
 *   Memory.  Every tensor pointer is device memory owned by the caller.  The
 *     library allocates no device memory on any call that enqueues work: the
 *     calls that need scratch memory take a caller-owned workspace, whose size
 *     a *_workspace_bytes query gives, and fail with GL_ERR_WORKSPACE when it
 *     is missing or short.  (gl_lookahead_create and
 *     gl_lookahead_set_profiling create HIP events; nothing else is created.)
 *     The library keeps no pointer after a call returns.  Buffers must stay
 *     alive until the streams the work was enqueued on have finished it.
 *   Layout.  Row-major, channels last: features [B, N, C], keys [B, M, C],
 *     neighbour indices int32 [B, N, k], weights [Cout, 2C], bias [Cout].
 *     Base pointers of feature, key and weight tensors must be 16-byte
 *     aligned; C must be a multiple of 8 (bf16) or 4 (fp32).
 *   Numbers.  dt selects the storage type of features, keys, weights, bias
 *     and outputs: GL_F32 or GL_BF16.  Arithmetic is fp32 (bf16 x bf16
 *     products are exact in fp32); outputs are rounded once to dt (RNE).
 *   Errors.  Arguments are validated on the host before anything is
 *     enqueued: a call either enqueues all of its work or none of it.  A
 *     failed launch returns GL_ERR_HIP.  Faults inside kernels surface at
 *     the caller's next synchronisation.  gl_last_error() gives a
 *     thread-local message for the last non-OK status.
 *   Streams.  hipStream_t may be 0 (the null stream).  Calls are
 *     asynchronous with respect to the host.  The library is thread-safe
 *     except that one lookahead handle must not be used from two threads
 *     at once.
 */
#ifndef GRAPHLEAP_H
#define GRAPHLEAP_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GL_VERSION 1
#define GL_MAX_KD 64     /* largest k * dilation of one graph build */
#define GL_MAX_M 4096    /* largest number of key nodes per image */
#define GL_MAX_K 64      /* largest neighbour count of one MRConv */

typedef enum gl_dtype { GL_F32 = 0, GL_BF16 = 1 } gl_dtype;

typedef enum gl_status {
  GL_OK = 0,
  GL_ERR_NULL_PTR = 1,     /* a required pointer is NULL */
  GL_ERR_BAD_SHAPE = 2,    /* a size is < 1, inconsistent or too large */
  GL_ERR_BAD_K = 3,        /* k < 1, dilation < 1, k*dilation > M or > GL_MAX_KD */
  GL_ERR_UNSUPPORTED = 4,  /* dtype, or C not a multiple of the vector width */
  GL_ERR_ALIGNMENT = 5,    /* a tensor base pointer is not 16-byte aligned */
  GL_ERR_ALIAS = 6,        /* an output overlaps an input it must not overlap */
  GL_ERR_HIP = 7,          /* the HIP runtime reported an error */
  GL_ERR_BAD_HANDLE = 8,   /* NULL or destroyed lookahead handle */
  GL_ERR_WORKSPACE = 9     /* a needed workspace is NULL, too small or misaligned */
} gl_status;

typedef enum gl_schedule {
  GL_SCHED_LOOKAHEAD = 0,        /* GraphLeap: block l uses G(X^(l-1)); the build of the
                                    next graph runs on the build stream while the update
                                    runs on the update stream */
  GL_SCHED_STANDARD = 1,         /* standard ViG (Eq. 6): block l uses G(X^l); build then
                                    update, serial, on the update stream */
  GL_SCHED_LOOKAHEAD_FUSED = 2   /* GraphLeap in one launch per block: the build tiles of
                                    the next graph and the update tiles of this block share
                                    one grid on the update stream (bit-identical results) */
} gl_schedule;

/* ---------------------------------------------------------------------------
 * gl_knn_graph -- dilated kNN graph (Sec. II-B Eq. 4; Sec. IV-B; Alg. 2).
 *
 * For every image b and query row i of x[b], ranks the key rows j of
 * keys[b] by the squared Euclidean distance between the L2-normalised rows
 * (norm floored at 1e-12), ties going to the lower j, keeps the
 * K' = k * dilation nearest and writes ranks 0, d, 2d, ..., (k-1)d:
 *     idx_out[b, i, t] = j of rank t * dilation,   t = 0 .. k-1.
 * Position 0 is the nearest key (the node itself when keys == x and rows
 * are distinct).  Distances are ranked at fixed-point resolution
 * 2^-(30 - ceil(log2 M)) (4e-6 at M = 4096, 2.4e-7 at M = 196); keys closer
 * than that count as tied and go to the lower index.
 *
 *   x       [B, N, C] queries (dt).
 *   keys    [B, M, C] keys (dt), or NULL for keys = x (then M must equal N).
 *   idx_out [B, N, k] int32 output; must not overlap x or keys.
 * Limits: B, N, C >= 1; 1 <= M <= GL_MAX_M; 1 <= k; 1 <= dilation;
 *         k * dilation <= min(M, GL_MAX_KD).
 * -------------------------------------------------------------------------*/
gl_status gl_knn_graph(const void* x, int B, int N, int C, const void* keys, int M,
                       int k, int dilation, gl_dtype dt, int32_t* idx_out,
                       hipStream_t stream);

/* ---------------------------------------------------------------------------
 * gl_pool_keys -- r x r average pooling of the H x W node grid, used as the
 * key set of the pyramid-stage workloads (a smaller key set for the kNN
 * graph of each node; the paper's own reduction between stages is the max
 * pooling of gl_max_pool_nodes, Sec. IV-E).
 *
 *   keys_out[b, p*(W/r) + q, c] = mean_{u,v<r} x[b, (p*r+u)*W + (q*r+v), c]
 * accumulated in fp32 and rounded once to dt.
 *   x [B, H*W, C] (dt); keys_out [B, (H/r)*(W/r), C] (dt), must not overlap x.
 * Limits: H % r == 0, W % r == 0, r >= 1.
 * -------------------------------------------------------------------------*/
gl_status gl_pool_keys(const void* x, int B, int H, int W, int C, int r, gl_dtype dt,
                       void* keys_out, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * gl_max_pool_nodes -- node reduction between the stages of a pyramid model:
 * r x r max pooling of the H x W node grid, stride r (Sec. IV-E: node counts
 * are reduced between stages by max pooling; r = 2 halves each grid side).
 * The width change that follows a stage boundary is a gl_linear projection.
 *
 *   out[b, p*(W/r) + q, c] = max_{u,v<r} x[b, (p*r+u)*W + (q*r+v), c]
 * exactly (a maximum of stored values needs no rounding).
 *   x [B, H*W, C] (dt), row-major grid; out [B, (H/r)*(W/r), C] (dt), must not
 *   overlap x.  Caller owns both (device memory); enqueued on `stream`.
 * Errors: GL_ERR_NULL_PTR, GL_ERR_UNSUPPORTED (dtype, C not a multiple of 8
 * (bf16) or 4 (fp32)), GL_ERR_BAD_SHAPE, GL_ERR_ALIGNMENT (16 bytes),
 * GL_ERR_ALIAS, GL_ERR_HIP.
 * Limits: H % r == 0, W % r == 0, r >= 1.
 * -------------------------------------------------------------------------*/
gl_status gl_max_pool_nodes(const void* x, int B, int H, int W, int C, int r, gl_dtype dt,
                            void* out, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * gl_mrconv -- max-relative graph convolution (Sec. II-A Eq. 2 and Eq. 3),
 * the feature update of one block.
 *
 *   m[b,i,c]   = max_t keys[b, idx[b,i,t], c] - x[b,i,c]
 *   out[b,i,o] = sum_c x[b,i,c] W[o,c] + sum_c m[b,i,c] W[o,C+c] + bias[o]
 * i.e. [x_i, max_j(x_j - x_i)] W^T + b with W = [W_x | W_m] (Sec. IV-C2).
 * The neighbour rows are gathered on the fly; no [B,N,k,C] edge tensor is
 * ever written.  Narrow layers gather straight into an on-chip tile and never
 * write the [B,N,2C] concatenation either.  When W is large per node (more
 * than 8 KB of W per node of the fused tile, e.g. C = Cout = 640) the call
 * runs two passes instead: the gather writes [x_i, m_i] rows to the caller's
 * workspace (B*N*2C*s bytes), then a tiled GEMM reads them.
 * gl_mrconv_workspace_bytes() gives the size (0 when the fused tile is used;
 * workspace may then be NULL).  A NULL, short or not 16-byte aligned
 * workspace where one is needed returns GL_ERR_WORKSPACE; it must not overlap
 * any other argument (GL_ERR_ALIAS).  The workspace is scratch: its contents
 * before and after the call do not matter, and two calls in flight at once
 * need two workspaces.
 *
 *   x    [B, N, C] (dt); keys [B, M, C] (dt) or NULL for keys = x (M == N).
 *   idx  [B, N, k] int32 in [0, M).  Out-of-range values are clamped into
 *        [0, M) inside the kernel (no fault; the result is then undefined).
 *   W    [Cout, 2C] (dt); bias [Cout] (dt) or NULL for zero bias.
 *   out  [B, N, Cout] (dt); must not overlap x, keys, idx, W or bias.
 * Limits: 1 <= k <= GL_MAX_K; Cout >= 1; one image's keys M * C * s bytes
 * below 32 GiB (2^31 16-byte vectors), else GL_ERR_BAD_SHAPE.
 * -------------------------------------------------------------------------*/
size_t gl_mrconv_workspace_bytes(int B, int N, int C, int k, int Cout, gl_dtype dt);
gl_status gl_mrconv(const void* x, int B, int N, int C, const void* keys, int M,
                    const int32_t* idx, int k, const void* W, const void* bias, int Cout,
                    gl_dtype dt, void* out, void* workspace, size_t workspace_bytes,
                    hipStream_t stream);

/* ---------------------------------------------------------------------------
 * gl_mrconv_noalloc -- gl_mrconv for callers that cannot allocate memory or
 * pass a workspace: code under HIP graph capture, serving loops and harnesses
 * that forbid allocation.  Same operation, arguments, layout and errors as
 * gl_mrconv, without the workspace.  The two-pass form's [x_i, m_i] rows go
 * to a buffer inside the library, GL_NOALLOC_SCRATCH_BYTES per device, which
 * a device holds from the library's load until the process ends; a layer
 * whose gl_mrconv_workspace_bytes() exceeds it fails with GL_ERR_WORKSPACE
 * before anything is enqueued.  The call itself allocates nothing.  Every
 * call on one device shares that buffer and it keeps the last call's rows:
 * calls that can overlap on one device (several streams or threads) race,
 * and the caller must order them.  `stream` must belong to the current
 * device (GL_ERR_UNSUPPORTED otherwise).
 * -------------------------------------------------------------------------*/
#define GL_NOALLOC_SCRATCH_BYTES (32u << 20)   /* 32 MiB */
gl_status gl_mrconv_noalloc(const void* x, int B, int N, int C, const void* keys, int M,
                            const int32_t* idx, int k, const void* W, const void* bias, int Cout,
                            gl_dtype dt, void* out, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * gl_mrconv_heads -- the multi-head MRConv update (Sec. II-A; per-head
 * W_x,h / W_m,h of Sec. IV-C2): channels split into `heads` equal contiguous
 * heads of hd = C / heads, and output head h sees only head h's channels of
 * x_i and of m_i:
 *   out[b,i,h*hd + o] = sum_{c<hd} x[b,i,h*hd+c] Wh[h,o,c]
 *                     + sum_{c<hd} m[b,i,h*hd+c] Wh[h,o,hd+c] + bias[h*hd+o]
 * Wh: [heads, hd, 2*hd] row-major in dt, head h's [W_x,h | W_m,h]; only the
 * heads' own weights are stored and read.  Cout == C.
 * hd a multiple of 4, at most 256 (bf16) / 128 (fp32), and the fused tile
 * fits LDS: the per-head kernel contracts each head's 2*hd channels on MFMA
 * (fp32 accumulation, one rounding) and needs no workspace.  Other head
 * widths: Wh is expanded into the dense block-diagonal [C, 2C] in the
 * workspace and the dense update runs on it.  heads == 1 is gl_mrconv with
 * W = Wh[0].
 * workspace: gl_mrconv_heads_workspace_bytes(B, N, C, k, heads, dt) bytes
 * (0: none needed), 16-byte aligned, disjoint from every other argument.
 * Everything else is as gl_mrconv.
 * Limits: heads >= 1, C % heads == 0.
 * -------------------------------------------------------------------------*/
size_t gl_mrconv_heads_workspace_bytes(int B, int N, int C, int k, int heads, gl_dtype dt);
gl_status gl_mrconv_heads(const void* x, int B, int N, int C, const void* keys, int M,
                          const int32_t* idx, int k, const void* Wh, const void* bias, int heads,
                          gl_dtype dt, void* out, void* workspace, size_t workspace_bytes,
                          hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Lookahead handle (Sec. IV-A, IV-F; the look-ahead buffer of Sec. IV-G).
 * Holds two HIP events that order the build stream against the update
 * stream; the caller owns both streams, every tensor and the workspace of
 * the layers that take the two-pass MRConv (see gl_mrconv).  Streams must be
 * distinct for the build to overlap the update; they may be equal.
 * -------------------------------------------------------------------------*/
typedef struct gl_lookahead* gl_lookahead_t;

/* Workspace bytes gl_graphleap_block / gl_graphleap_stack need for blocks of
 * this shape (the MRConv workspace of gl_mrconv with Cout = C, keys pooled
 * r x r when pool_r > 1); 0 when none is needed or the shape is invalid. */
size_t gl_graphleap_workspace_bytes(int B, int H, int W, int C, int pool_r, int k, gl_dtype dt);

gl_status gl_lookahead_create(hipStream_t s_update, hipStream_t s_build, gl_lookahead_t* out);
gl_status gl_lookahead_destroy(gl_lookahead_t h);

/* Profiling: when enabled (max_records > 0), every kNN build, MRConv update
 * and one-launch block enqueued through the handle is stamped by its own
 * dispatch with a start and an end HIP event (at most max_records pairs of
 * each kind are kept; later launches are not timed).
 * gl_lookahead_kernel_times() synchronises the recorded events of one kind
 * (which = GL_TIME_BUILD, GL_TIME_UPDATE, GL_TIME_FUSED or GL_TIME_LINEAR),
 * writes their
 * durations in milliseconds (at most cap of them) and clears that kind's
 * records.  max_records == 0 disables it. */
#define GL_TIME_BUILD 0
#define GL_TIME_UPDATE 1
#define GL_TIME_FUSED 2   /* one-launch blocks of GL_SCHED_LOOKAHEAD_FUSED */
#define GL_TIME_LINEAR 3  /* fully connected layers of the full ViG block */
gl_status gl_lookahead_set_profiling(gl_lookahead_t h, int max_records);
gl_status gl_lookahead_kernel_times(gl_lookahead_t h, int which, float* ms_out, int cap,
                                    int* n_out);

/* Bootstrap Ghat^0 = G(X^0) with dilation d_0 (Sec. III: the first block
 * uses the standard construction).  Enqueues [pooling of x0 into keys_ws on
 * the update stream when pool_r > 1], then the build into idx0 on the build
 * stream after the update stream's prior work; the next gl_graphleap_block
 * waits for it.  x0 [B, H*W, C]; keys_ws [B, (H/pool_r)*(W/pool_r), C] or
 * NULL when pool_r == 1; idx0 [B, H*W, k]. */
gl_status gl_lookahead_bootstrap(gl_lookahead_t h, const void* x0, int B, int H, int W,
                                 int C, int pool_r, void* keys_ws, int k, int dilation0,
                                 gl_dtype dt, int32_t* idx0);

/* ---------------------------------------------------------------------------
 * gl_graphleap_block -- one GraphLeap block in the reduced form
 * X^(l+1) = MRConv(X^l; Ghat^l) (Eq. 12-13 with U = X), overlapping the
 * build of Ghat^(l+1) = G(X^l) (Eq. 11 for the next block) with the update.
 *
 * Enqueue order:
 *   update stream: wait for the previous build through the handle (it made
 *                  idx_use); [pool x_in -> keys_ws]; record "x_in ready";
 *   build stream : wait "x_in ready"; kNN(x_in, keys) -> idx_next with
 *                  dilation_next; record "built" (skipped if idx_next NULL);
 *   update stream: MRConv(x_in, keys, idx_use, Wt, bias) -> x_out.
 * Both engines read only x_in (and keys_ws), so they run concurrently.
 *
 *   x_in [B, H*W, C]; x_out [B, H*W, C] must not overlap x_in, keys_ws.
 *   keys_ws [B, M, C] with M = (H/pool_r)*(W/pool_r) when pool_r > 1,
 *           else NULL (keys = x_in).
 *   idx_use [B, H*W, k] = Ghat^l; idx_next [B, H*W, k] = Ghat^(l+1) or NULL
 *           (last block, or when Ghat^(l+1) is the same graph as Ghat^l);
 *           idx_next must not overlap idx_use.
 *   Wt [C, 2C], bias [C] or NULL.
 *   workspace: at least gl_graphleap_workspace_bytes() bytes (may be NULL
 *           when that is 0); used on the update stream only.
 * The caller double-buffers features and graphs (two of each, Sec. IV-G
 * N_buf = 2): the handle's waits make reuse of the buffers of block l-1 by
 * block l+1 safe.
 * -------------------------------------------------------------------------*/
gl_status gl_graphleap_block(gl_lookahead_t h, const void* x_in, int B, int H, int W, int C,
                             int pool_r, void* keys_ws, const int32_t* idx_use, int k,
                             const void* Wt, const void* bias, gl_dtype dt, void* x_out,
                             int32_t* idx_next, int dilation_next, void* workspace,
                             size_t workspace_bytes);

/* ---------------------------------------------------------------------------
 * gl_graphleap_stack -- L blocks of X^(l+1) = MRConv(X^l; Ghat^l) enqueued
 * natively (Alg. 1 reduced to graph + MRConv, looped over blocks).
 *
 *   schedule GL_SCHED_LOOKAHEAD: Ghat^0 = G(X^0, d_0); Ghat^1 = G(X^0, d_1)
 *     (the same graph when d_1 == d_0, built once); Ghat^l = G(X^(l-1), d_l)
 *     for l >= 2, each built on the build stream while the previous block
 *     updates.  L - 1 builds when d_1 == d_0; G(X^(L-1)) is never built.
 *   schedule GL_SCHED_STANDARD: Ghat^l = G(X^l, d_l), build then update,
 *     all on the update stream (Eq. 5-7 with U = X).
 *   schedule GL_SCHED_LOOKAHEAD_FUSED: the lookahead graphs as above, but each
 *     block is one launch on the update stream whose grid holds both the
 *     build tiles of Ghat^(l+1) and the update tiles of X^(l+1) (for updates
 *     in the two-pass form, the gather tiles, with the GEMM pass launched
 *     next; builds over large key sets run as their own launch first); the
 *     results are bit-identical to GL_SCHED_LOOKAHEAD.
 *
 *   x0 [B, N, C] input, N = H*W.  Ws [L, C, 2C]; bs [L, C] or NULL.
 *   dilations: host array of L ints (the dilation of the block that uses
 *     each graph).
 *   x_ws [2, B, N, C] feature ping-pong workspace; idx_ws [2, B, N, k];
 *   keys_ws [B, M, C] when pool_r > 1 else NULL;  x_out [B, N, C] = X^L.
 *   workspace: at least gl_graphleap_workspace_bytes() bytes (NULL when 0).
 *   x_out, x_ws, idx_ws, keys_ws and workspace must not overlap each other
 *   or x0.  Every block is checked before anything is enqueued.
 * -------------------------------------------------------------------------*/
gl_status gl_graphleap_stack(gl_lookahead_t h, const void* x0, int B, int H, int W, int C,
                             int pool_r, int L, int k, const int* dilations, const void* Ws,
                             const void* bs, gl_dtype dt, gl_schedule schedule, void* x_ws,
                             int32_t* idx_ws, void* keys_ws, void* x_out, void* workspace,
                             size_t workspace_bytes);

/* ---------------------------------------------------------------------------
 * Diagnostics.
 * -------------------------------------------------------------------------*/
const char* gl_status_string(gl_status s);
const char* gl_last_error(void);   /* thread-local detail of the last non-OK status */
int gl_version(void);

/* ===========================================================================
 * The full GraphLeap ViG block (Sec. III Eq. 11-15, Alg. 1): FC1, the
 * leap-ahead graph, MRConv, FC2 + residual and the FFN + residual.
 * ========================================================================= */

typedef enum { GL_ACT_NONE = 0, GL_ACT_GELU = 1 } gl_act;

/* ---------------------------------------------------------------------------
 * gl_linear -- one fully connected layer over the channel axis (FC1, FC2 and
 * the FFN of Eq. 11, 14, 15):
 *   out[r, o] = act_out( sum_c act_in(x[r, c]) W[o, c] + bias[o] ) + residual[r, o]
 * act = GL_ACT_GELU is the exact GELU x Phi(x); act_in is applied to x's
 * stored values and rounded back to dt (as if sigma(x) had been stored),
 * everything after the contraction is fp32, rounded once to dt.
 *   x [R, K] (dt); W [Cout, K] (dt); bias [Cout] (dt) or NULL;
 *   residual [R, Cout] (dt) or NULL, and may be `out` itself (in place);
 *   out [R, Cout] (dt), must not overlap x, W or bias.
 * Limits: R, K, Cout >= 1; K % 8 == 0 (bf16) or K % 4 == 0 (fp32).
 * -------------------------------------------------------------------------*/
gl_status gl_linear(const void* x, int R, int K, const void* W, const void* bias, int Cout,
                    gl_act act_in, gl_act act_out, const void* residual, gl_dtype dt,
                    void* out, hipStream_t stream);

/* Weights of one full block (dt, row-major [out, in]; biases may be NULL). */
typedef struct {
  const void* W_in;   /* [C, C]   FC1 */
  const void* b_in;   /* [C] */
  const void* W_upd;  /* [C, 2C]  MRConv update, [W_x | W_m] */
  const void* b_upd;  /* [C] */
  const void* W_out;  /* [C, C]   FC2 */
  const void* b_out;  /* [C] */
  const void* W_1;    /* [4C, C]  FFN hidden layer */
  const void* b_1;    /* [4C] */
  const void* W_2;    /* [C, 4C]  FFN output layer */
  const void* b_2;    /* [C] */
} gl_vig_params;

/* Bytes of the workspace gl_vig_block and gl_vig_stack need for an H x W
 * node grid (N = H*W) whose keys are pooled pool_r x pool_r (1: none).  They
 * carve sigma(U~), Y, the FFN's hidden rows (that region also serves the
 * two-pass MRConv) and the pooled keys of U out of it, and the stack also U,
 * two feature buffers and two graphs.  0 when the shape is invalid. */
size_t gl_vig_workspace_bytes(int B, int H, int W, int C, int pool_r, int k, gl_dtype dt);

/* ---------------------------------------------------------------------------
 * gl_vig_block -- one full block on the lookahead handle's streams, given the
 * graph it uses (Alg. 1):
 *   U = x_in W_in^T + b_in -> u_out           (cached for the next graph)
 *   [pool_r > 1: keys = U pooled pool_r x pool_r over the H x W grid
 *    (M = (H/pool_r)*(W/pool_r) rows, in ws); else keys = U, M = N]
 *   [build idx_next = G(U, keys, dilation_next) on the build stream,
 *    overlapping everything below; skipped when idx_next is NULL]
 *   Ut = MRConv(U; keys, idx_use)  (W_upd, b_upd)
 *   Y = GELU(Ut) W_out^T + b_out + x_in
 *   x_out = GELU(Y W_1^T + b_1) W_2^T + b_2 + Y
 * Every GELU is taken in fp32 before its output is rounded to dt: MRConv
 * stores GELU(Ut), FFN1 stores GELU(Y W_1^T + b_1).
 * Key pooling is the pyramid stages' (Sec. IV-E), as in gl_graphleap_block.
 * Enqueues on the update stream after waiting for the handle's previous
 * build.  x_in, x_out, u_out [B, N, C]; idx_use, idx_next [B, N, k] int32
 * indexing the M keys; ws of at least gl_vig_workspace_bytes(), 256-byte
 * aligned.  The build of idx_next reads u_out and the keys in ws; the next
 * block enqueued through the handle waits for it before it writes either.
 * x_out must not overlap x_in, u_out, ws or the graphs.
 * Limits: H % pool_r == 0 and W % pool_r == 0, k <= M; the kNN and MRConv
 * limits of gl_knn_graph and gl_mrconv.
 * -------------------------------------------------------------------------*/
gl_status gl_vig_block(gl_lookahead_t h, const void* x_in, int B, int H, int W, int C, int pool_r,
                       int k, const int32_t* idx_use, const gl_vig_params* p, gl_dtype dt,
                       void* ws, size_t ws_bytes, void* u_out, int32_t* idx_next,
                       int dilation_next, void* x_out);

/* ---------------------------------------------------------------------------
 * gl_vig_stack -- L full blocks, natively enqueued.
 *   GL_SCHED_LOOKAHEAD: Ghat^0 = G(U^0, d_0), Ghat^l = G(U^(l-1), d_l)
 *     (Eq. 12 and Alg. 1's bootstrap); each build runs on the build stream
 *     while the rest of its block runs on the update stream.
 *   GL_SCHED_LOOKAHEAD_FUSED: the same graphs; one stream, each build in one
 *     launch with its block's MRConv, or with the gather pass of a two-pass
 *     MRConv (both read only U^l); builds over large key sets run alone.
 *   GL_SCHED_STANDARD: Ghat^l = G(U^l, d_l) (Eq. 6), serial.
 * With pool_r > 1 each graph ranks the keys pooled from the U it is built
 * from and each MRConv gathers the keys pooled from its own U (as
 * gl_vig_block).  params: L blocks' weights.  x0, x_out [B, H*W, C]; ws of
 * at least gl_vig_workspace_bytes(), 256-byte aligned; x_out must not overlap
 * x0 or ws.  Every block is checked before anything is enqueued.
 * -------------------------------------------------------------------------*/
gl_status gl_vig_stack(gl_lookahead_t h, const void* x0, int B, int H, int W, int C, int pool_r,
                       int L, int k, const int* dilations, const gl_vig_params* params,
                       gl_dtype dt, gl_schedule schedule, void* ws, size_t ws_bytes,
                       void* x_out);

#ifdef __cplusplus
}
#endif

#endif /* GRAPHLEAP_H */
