/*
 * libgspn -- GSPN 2D line-scan propagation on AMD Instinct MI355X (gfx950).
 *
 * The operation (Sec. 3 of "Scaling Parallel Sequence Models to
 * Foundation-Scale Vision Encoders", Eqs. (gspn_recurrence), (gspn_output),
 * (row_stochastic_norm); channel-shared weights as in Sec. 4.2, Eq. (2dsp)):
 *
 *   for every direction d in the mask, batch b and channel c (group g = c/(C/G)),
 *   scanning the lines i = 0..L-1 of the grid in direction d:
 *
 *     h_i[j] = sum_{k=0..2} w_d[b,g,k @ (i,j)] * h_{i-1}[j+k-1]
 *              + lam_d[b,c @ (i,j)] * x[b,c @ (i,j)]          (h_{-1} = 0)
 *     y[b,c @ (i,j)] = sum_d u_d[b,c @ (i,j)] * h_i[j]
 *
 *   "@ (i,j)" is the pixel at step i, line position j of direction d:
 *     top-to-bottom (i, j)   bottom-to-top (H-1-i, j)
 *     left-to-right (j, i)   right-to-left (j, W-1-i)     as (row, col).
 *   Tap k at a pixel reads the previous line at perpendicular offset k-1
 *   (column offset for vertical scans, row offset for horizontal ones), i.e.
 *   the "top-left, top-center, top-right" neighbours of Sec. 3.  Taps that
 *   leave the grid and all taps on the first scanned line are ignored (any
 *   value, NaN included); their gradients are written as 0.
 *
 * Storage and arithmetic: every tensor of one call has the same storage type
 * (fp32 or bf16); arithmetic is fp32 and results are rounded to the storage
 * type (round to nearest even) once, when stored.
 *
 * Layouts.  D = number of directions in the mask; per-direction tensors are
 * stacked in increasing direction-bit order.  The entry points without a
 * suffix take every tensor pixel-major (row-major images):
 *   x, y, dy, dx           [B][C][H][W]          element (r, c) at r*W + c
 *   lam, u, dlam, du       [D][B][C][H][W]
 *   w, dw                  [D][B][G][3][H][W]    tap k of pixel (r, c)
 * The _blocked entry points take the per-direction tensors in the order in
 * which their direction scans them ("blocked line-major"): the lines a
 * direction scans (storage rows for vertical scans, storage columns for
 * horizontal ones) are grouped in blocks of 8 consecutive lines, and inside a
 * block the 8 values of one line position are adjacent:
 *   lam, u, dlam, du       [D][B][C][plane]
 *   w, dw                  [D][B][G][3][plane]
 *   plane of L lines of P positions, line l, position p at
 *       8*P*(l/8) + n*p + l%8,   n = min(8, L - 8*(l/8))
 *   vertical direction (T2B, B2T):    line = row r, position = column c,
 *                                     L = H, P = W
 *   horizontal direction (L2R, R2L):  line = column c, position = row r,
 *                                     L = W, P = H
 * (the last block holds L%8 lines when L is not a multiple of 8; a plane
 * has exactly H*W elements).  A producer of lam, u and w (for instance the
 * 1x1 convolutions that predict them) can write this layout directly; the
 * kernels then read every stream with whole-line accesses.  x, y, dy and dx
 * are pixel-major in both.
 *
 * Ownership and threading: all pointers are device pointers owned by the
 * caller; the library keeps none of them after a call returns, allocates no
 * memory and holds no state between calls.  Outputs are fully overwritten
 * (never accumulated into); inputs are never written.  Buffers of one call
 * must not overlap.  Every base pointer must be 16-byte aligned.  Calls are
 * asynchronous on `stream` (a hipStream_t; NULL is the null stream), launch
 * only on that stream and never synchronise the device.  Calls are
 * thread-safe.
 *
 * Workspace: some shapes need device memory beyond their inputs and outputs
 * (partial sums of a weight group split over several workgroups, per-direction
 * fp32 planes of long lines, the normalized weights of the _norm entry points,
 * the latent tensors of gspn_latent_fwd).  The caller provides it:
 * gspn_workspace_size (gspn_latent_workspace_size) gives the bytes a call
 * takes for its sizes; the call takes `workspace` (16-byte aligned, not
 * overlapping any other buffer of the call; may be NULL when the size is 0)
 * and its size `workspace_bytes`, and returns GSPN_ERR_WORKSPACE when it is
 * smaller than needed.  The workspace's contents on entry do not matter and
 * are undefined after the call; calls that share a workspace must not run
 * concurrently.
 *
 * Errors: every argument check runs on the host before any HIP call, so an
 * invalid call has no effect on the device.  A failed HIP call returns
 * GSPN_ERR_HIP (see gspn_last_hip_error).  No C++ exception crosses the ABI.
 */
#ifndef GSPN_H
#define GSPN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Scan directions (bitmask). */
#define GSPN_T2B 1
#define GSPN_B2T 2
#define GSPN_L2R 4
#define GSPN_R2L 8
#define GSPN_ALL 15

/* Storage types. */
#define GSPN_F32 0
#define GSPN_BF16 1

/* Status codes. */
#define GSPN_OK 0
#define GSPN_ERR_NULL (-1)        /* a required pointer is NULL                 */
#define GSPN_ERR_DIM (-2)         /* a size < 1, or C not a multiple of G       */
#define GSPN_ERR_DIRECTION (-3)   /* direction mask outside [1, 15]             */
#define GSPN_ERR_DTYPE (-4)       /* unknown storage type                       */
#define GSPN_ERR_ALIGN (-5)       /* a base pointer is not 16-byte aligned      */
#define GSPN_ERR_ALIAS (-6)       /* two buffers of the call overlap            */
#define GSPN_ERR_UNSUPPORTED (-7) /* H or W > GSPN_MAX_SIDE, or too many elements */
#define GSPN_ERR_HIP (-8)         /* a HIP runtime call or launch failed        */
#define GSPN_ERR_WORKSPACE (-9)   /* workspace (or reserve) missing or too small */

/* Operations, for gspn_workspace_size. */
#define GSPN_OP_FWD 0
#define GSPN_OP_BWD 1
#define GSPN_OP_FWD_NORM 2
#define GSPN_OP_BWD_NORM 3
#define GSPN_OP_FWD_BLOCKED 4
#define GSPN_OP_BWD_BLOCKED 5
#define GSPN_OP_FWD_TRAIN 6
#define GSPN_OP_BWD_RESERVE 7
#define GSPN_OP_FWD_NORM_TRAIN 8
#define GSPN_OP_BWD_NORM_RESERVE 9

/* Largest supported H and W, and largest B*C*H*W and B*G*H*W*3*D. */
#define GSPN_MAX_SIDE 4096
#define GSPN_MAX_ELEMS (((int64_t)1) << 40)

/*
 * Bytes of workspace that operation `op` (GSPN_OP_*) takes for these sizes,
 * in *bytes (0 for most shapes).  The same argument checks as the call; the
 * plan of a call is the same for every call with these sizes on one device.
 * Needs the current device (GSPN_ERR_HIP without one).
 */
int gspn_workspace_size(int op, int direction, int B, int C, int G, int H, int W, int dtype,
                        int64_t *bytes);

/*
 * Forward pass (Sec. 3, Eqs. (gspn_recurrence) and (gspn_output)).
 *   x    [B][C][H][W]        input feature map
 *   w    [D][B][G][3][H][W]  neighbour weights (normalised, e.g. row-stochastic)
 *   lam  [D][B][C][H][W]     input scaling lambda_d
 *   u    [D][B][C][H][W]     output gate u_d
 *   y    [B][C][H][W]        out: sum over directions of u_d * h_d
 *   direction  bitmask of GSPN_T2B | GSPN_B2T | GSPN_L2R | GSPN_R2L
 *   G          weight groups; channel c uses group c / (C/G); C % G == 0
 *              (G = 1 is Eq. (2dsp) of Sec. 4.2, G = C Eq. (gspn_recurrence))
 *   dtype      GSPN_F32 or GSPN_BF16 (all tensors)
 *   workspace, workspace_bytes   see "Workspace" above
 *   stream     hipStream_t to launch on
 * Returns GSPN_OK or a negative status.
 */
int gspn_scan_fwd(const void *x, const void *w, const void *lam, const void *u,
                  void *y, int direction, int B, int C, int G, int H, int W,
                  int dtype, void *workspace, int64_t workspace_bytes, void *stream);

/*
 * Backward pass: gradients of a loss l(y) given dy = dl/dy.  The backward of
 * the recurrence is not printed in the paper (which reports only its run
 * time); with the adjoint a_i = dl/dh_i it is
 *   a_i[j]  = u_i[j] dy_i[j] + sum_k w_{i+1}[j-k+1, k] a_{i+1}[j-k+1],  a_L = 0
 *   du_i    = dy_i * h_i,   dlam_i = a_i * x_i,   dx = sum_d a_d * lam_d,
 *   dw_i[j,k] = sum_{c in group} a_i[j] h_{i-1}[j+k-1]   (0 on ignored taps).
 * h is recomputed on the GPU; nothing is saved by the forward pass.
 *   dy   [B][C][H][W]        in: gradient of the merged output y
 *   dx   [B][C][H][W]        out
 *   dw   [D][B][G][3][H][W]  out
 *   dlam [D][B][C][H][W]     out
 *   du   [D][B][C][H][W]     out
 * Other arguments as in gspn_scan_fwd.
 */
int gspn_scan_bwd(const void *x, const void *w, const void *lam, const void *u,
                  const void *dy, void *dx, void *dw, void *dlam, void *du,
                  int direction, int B, int C, int G, int H, int W, int dtype,
                  void *workspace, int64_t workspace_bytes, void *stream);

/*
 * gspn_scan_fwd and gspn_scan_bwd with lam, u, w, dlam, du and dw in the
 * blocked line-major layout (see "Layouts" above), for producers that write
 * the per-direction tensors in their scan order.  Same operation, arguments,
 * checks and errors.
 */
int gspn_scan_fwd_blocked(const void *x, const void *w, const void *lam, const void *u,
                          void *y, int direction, int B, int C, int G, int H, int W,
                          int dtype, void *workspace, int64_t workspace_bytes, void *stream);
int gspn_scan_bwd_blocked(const void *x, const void *w, const void *lam, const void *u,
                          const void *dy, void *dx, void *dw, void *dlam, void *du,
                          int direction, int B, int C, int G, int H, int W, int dtype,
                          void *workspace, int64_t workspace_bytes, void *stream);

/*
 * The two passes with the weights given by their logits wt, laid out like w
 * (pixel-major): Sec. 3, Eq. (row_stochastic_norm) forms
 *   w(j,k) = sigma(wt(j,k)) / max(sum_{k' in N(j)} sigma(wt(j,k')), 1e-30)
 * with sigma the logistic sigmoid and N(j) the taps whose neighbour lies on
 * the grid (the others get weight 0; the clamp is a reading, the paper names
 * no constant).  Taps outside N(j) may hold any value.  The weights are
 * formed once per group and pixel, in fp32, and stored in the storage type in
 * the workspace for the scan.
 *   w_logits   [D][B][G][3][H][W]   in
 *   dw_logits  [D][B][G][3][H][W]   out (backward): dl/dwt, from dl/dw by
 *       dl/dwt_m = sigma(wt_m)(1 - sigma(wt_m)) (dw_m - sum_k w_k dw_k) / S
 *     on N(j) (S the clamped sum), 0 elsewhere; dl/dw passes through the
 *     storage type on the way.
 * Other arguments, checks and errors as in gspn_scan_fwd / gspn_scan_bwd.
 */
int gspn_scan_fwd_norm(const void *x, const void *w_logits, const void *lam,
                       const void *u, void *y, int direction, int B, int C,
                       int G, int H, int W, int dtype, void *workspace,
                       int64_t workspace_bytes, void *stream);

int gspn_scan_bwd_norm(const void *x, const void *w_logits, const void *lam,
                       const void *u, const void *dy, void *dx, void *dw_logits,
                       void *dlam, void *du, int direction, int B, int C, int G,
                       int H, int W, int dtype, void *workspace,
                       int64_t workspace_bytes, void *stream);

/*
 * Training pair: the forward and backward passes of gspn_scan_fwd and
 * gspn_scan_bwd (same operation, results bit for bit), where the forward
 * also leaves in a caller buffer, the reserve, what the backward of the same
 * inputs would otherwise have to make again from them -- the analogue of the
 * tensors an autograd forward saves for its backward.  On the bf16 square
 * planes of side 24 to 64 (multiples of 8) the backward reads the weights
 * and the horizontal directions' lambda and u as 16-byte pieces of 8 steps
 * of one line position; gspn_scan_bwd re-lays them out into that order
 * first, while gspn_scan_fwd_train writes those copies as it reads its
 * inputs and gspn_scan_bwd_reserve reads them from the reserve.
 *   gspn_reserve_size     bytes of the reserve for these sizes (0 where
 *                         the backward re-lays nothing out; the pair then
 *                         runs as the plain pair and reserve may be NULL)
 *   reserve               device buffer of at least that size, 16-byte
 *                         aligned, overlapping no other buffer of the call;
 *                         written by gspn_scan_fwd_train, read (not written)
 *                         by gspn_scan_bwd_reserve
 * The backward must get the x, w, lam and u that the forward which wrote the
 * reserve read, unchanged, and the reserve unchanged since; a mismatch is not
 * detected (the gradients are then those of the inputs the reserve came
 * from, mixed with the new ones).  GSPN_ERR_WORKSPACE when reserve is NULL or
 * reserve_bytes below the size.  Workspace: gspn_workspace_size with
 * GSPN_OP_FWD_TRAIN / GSPN_OP_BWD_RESERVE.  Other arguments, checks and
 * errors as in gspn_scan_fwd / gspn_scan_bwd.
 */
int gspn_reserve_size(int direction, int B, int C, int G, int H, int W, int dtype,
                      int64_t *bytes);
int gspn_scan_fwd_train(const void *x, const void *w, const void *lam, const void *u,
                        void *y, int direction, int B, int C, int G, int H, int W,
                        int dtype, void *reserve, int64_t reserve_bytes,
                        void *workspace, int64_t workspace_bytes, void *stream);
int gspn_scan_bwd_reserve(const void *x, const void *w, const void *lam, const void *u,
                          const void *dy, void *dx, void *dw, void *dlam, void *du,
                          int direction, int B, int C, int G, int H, int W, int dtype,
                          const void *reserve, int64_t reserve_bytes, void *workspace,
                          int64_t workspace_bytes, void *stream);

/*
 * The training pair of the _norm entry points (weights given as logits):
 * gspn_scan_fwd_norm and gspn_scan_bwd_norm, bit for bit, where the forward
 * keeps in the reserve the weights it forms from the logits (in the blocked
 * order, every direction) and the horizontal directions' lambda and u
 * copies, and the backward takes them from there instead of forming and
 * copying them again.  gspn_reserve_size_norm gives the reserve's bytes;
 * arguments, rules and errors otherwise as for gspn_scan_fwd_train /
 * gspn_scan_bwd_reserve and the _norm entry points (workspace:
 * gspn_workspace_size with GSPN_OP_FWD_NORM_TRAIN / GSPN_OP_BWD_NORM_RESERVE).
 */
int gspn_reserve_size_norm(int direction, int B, int C, int G, int H, int W, int dtype,
                           int64_t *bytes);
int gspn_scan_fwd_norm_train(const void *x, const void *w_logits, const void *lam,
                             const void *u, void *y, int direction, int B, int C, int G,
                             int H, int W, int dtype, void *reserve, int64_t reserve_bytes,
                             void *workspace, int64_t workspace_bytes, void *stream);
int gspn_scan_bwd_norm_reserve(const void *x, const void *w_logits, const void *lam,
                               const void *u, const void *dy, void *dx, void *dw_logits,
                               void *dlam, void *du, int direction, int B, int C, int G, int H,
                               int W, int dtype, const void *reserve, int64_t reserve_bytes,
                               void *workspace, int64_t workspace_bytes, void *stream);

/*
 * gspn_scan_bwd for callers that cannot allocate device memory or hand in a
 * workspace: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Same operation, arguments (without the workspace), checks
 * and errors as gspn_scan_bwd; its workspace is a fixed device array of
 * GSPN_STATIC_SCRATCH_BYTES that the library holds on every GPU it runs on
 * until the process ends (looked up, not allocated, at the first call on a
 * device).  Returns GSPN_ERR_WORKSPACE, before any launch, when the call
 * needs more (gspn_workspace_size with GSPN_OP_BWD gives the need).  Every
 * call on one GPU shares that GPU's array: calls that overlap in time on one
 * GPU (concurrent streams or threads) race and must not be issued; calls
 * ordered on one stream are safe.  Allocates nothing, not even through
 * another library.
 */
#define GSPN_STATIC_SCRATCH_BYTES (((int64_t)64) << 20)
int gspn_scan_bwd_static(const void *x, const void *w, const void *lam, const void *u,
                         const void *dy, void *dx, void *dw, void *dlam, void *du,
                         int direction, int B, int C, int G, int H, int W, int dtype,
                         void *stream);

/*
 * gspn_scan_bwd with the launch plan of the register-streamed backward (the
 * bf16 kernels for square planes whose side is a multiple of 8 from 24 to
 * 64, groups of more than one channel) fixed by the caller, for tests of determinism across
 * launch shapes and for tuning.  That backward takes the channels of a group
 * in workgroups of up to `slots` channels, one step's weight-gradient terms
 * summed over them in LDS, the workgroups' fp32 partials summed afterwards:
 *   slots  0   the library's choice (the same plan as gspn_scan_bwd)
 *          4   workgroups of 4 channels, where a group has at least 4
 *          8   workgroups of up to 8 channels (as many as fit in LDS)
 * A plan the shape cannot take, and every other kernel family, run as in
 * gspn_scan_bwd.  dx, dlam and du do not depend on the plan (bit for bit);
 * dw is summed over a group's channels in another association, so it may
 * differ in the last bit of the fp32 sum before its one rounding.
 * gspn_workspace_size_slots gives the workspace of that plan.  Other
 * values of slots: GSPN_ERR_UNSUPPORTED.  Other arguments, checks and
 * errors as in gspn_scan_bwd.
 */
int gspn_workspace_size_slots(int slots, int direction, int B, int C, int G, int H, int W,
                              int dtype, int64_t *bytes);
int gspn_scan_bwd_slots(int slots, const void *x, const void *w, const void *lam,
                        const void *u, const void *dy, void *dx, void *dw, void *dlam,
                        void *du, int direction, int B, int C, int G, int H, int W,
                        int dtype, void *workspace, int64_t workspace_bytes, void *stream);

/*
 * Latent-space propagation sublayer of C-GSPN (Sec. 5, Eqs. (latent_down),
 * (latent_params), (latent_recurrence), (latent_up)): the feature map is
 * projected per pixel from C to Cc channels, the propagation parameters are
 * predicted per pixel from the latent map, the four-direction scan runs on
 * the Cc latent channels with one weight group per channel (G = Cc), and the
 * result is projected back to C channels:
 *   x_c   = P_down x                        [B][Cc][H][W]
 *   u_d   = L_u,d x_c,  lam_d = L_lam,d x_c  (per direction d of the mask)
 *   wt_d  = L_w,d x_c   (three tap logits per latent channel and pixel)
 *   w_d   = row-stochastic weights from wt_d (as in gspn_scan_fwd_norm)
 *   y_c   = scan(x_c, w, lam, u)             (gspn_scan_fwd, G = Cc)
 *   y     = P_up y_c                         [B][C][H][W]
 * The paper fixes neither biases nor activations on u and lambda: the
 * projections here are linear without bias.  Storage is bf16 only
 * (dtype GSPN_BF16; GSPN_F32 is GSPN_ERR_UNSUPPORTED); products accumulate in
 * fp32 on the matrix cores.  x_c, u, lam, w and y_c are stored in bf16
 * between the stages, in the workspace (gspn_latent_workspace_size gives its
 * size); the logits wt are normalized in registers and never stored.
 * Weight layouts (row-major, output channel first):
 *   p_down [Cc][C]      l_u, l_lam [D][Cc][Cc]      l_w [D][Cc][3][Cc]
 *   p_up   [C][Cc]      (row (c, k) of l_w gives the logit of tap k of
 *                        latent channel c)
 * C and Cc must be multiples of 8 (GSPN_ERR_UNSUPPORTED otherwise).  Other
 * arguments, checks and errors as in gspn_scan_fwd.
 */
int gspn_latent_workspace_size(int direction, int B, int C, int Cc, int H, int W,
                               int dtype, int64_t *bytes);
int gspn_latent_fwd(const void *x, const void *p_down, const void *l_u,
                    const void *l_lam, const void *l_w, const void *p_up, void *y,
                    int direction, int B, int C, int Cc, int H, int W, int dtype,
                    void *workspace, int64_t workspace_bytes, void *stream);
/*
 * The two kinds of stage of gspn_latent_fwd, for callers that keep the
 * latent tensors themselves.
 * gspn_project: the per-pixel projection (1x1 convolution) of Eqs.
 * (latent_down) and (latent_up), y[b] = a x[b]:
 *   a [M][K], x [B][K][H][W], y [B][M][H][W]; K a multiple of 8; bf16.
 * gspn_latent_params: Eq. (latent_params) with the weights normalized as in
 * Eq. (row_stochastic_norm), written in the blocked line-major layout of
 * gspn_scan_fwd_blocked (G = Cc):
 *   xc [B][Cc][H][W] in; u, lam [D][B][Cc][plane], w [D][B][Cc][3][plane] out;
 *   Cc a multiple of 8; bf16.
 */
int gspn_project(const void *a, const void *x, void *y, int B, int M, int K,
                 int H, int W, int dtype, void *stream);
int gspn_latent_params(const void *xc, const void *l_u, const void *l_lam,
                       const void *l_w, void *u, void *lam, void *w,
                       int direction, int B, int Cc, int H, int W, int dtype,
                       void *stream);
/* Static description of a status code (never NULL). */
const char *gspn_strerror(int status);

/* hipError_t of the most recent GSPN_ERR_HIP on the calling thread (0 if none). */
int gspn_last_hip_error(void);

/* Library version as 10000*major + 100*minor + patch. */
int gspn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* GSPN_H */
