/*
 * gspn.h -- C ABI of the GSPN 2D line-scan propagation on AMD Instinct MI355X (gfx950).
 *
 * The operation (Generalized Spatial Propagation Network, Sec. 3.1 Eq. 1-2,
 * Sec. 3.3; supplementary Eq. 7-9):
 *
 *   For each (b, c) plane of an H x W map and each direction d of `mask`,
 *   lines (rows for T2B/B2T, columns for L2R/R2L) are visited in the
 *   direction's order.  With the state before the first line equal to zero,
 *
 *     h_d[line][p] = sum_{k=0..2} w_{d,k}[line][p] * h_d[prev line][p + k - 1]
 *                    + lam[line][p] * x[line][p]
 *
 *   where p is the position along the line and a neighbour outside the line
 *   contributes 0.  The output merges the directions by summation:
 *
 *     y = u * sum_d h_d
 *
 *   Neighbours (k = 0, 1, 2 is offset -1, 0, +1 along the line coordinate):
 *     T2B  rows 0..H-1   (i-1, j-1) (i-1, j) (i-1, j+1)
 *     B2T  rows H-1..0   (i+1, j-1) (i+1, j) (i+1, j+1)
 *     L2R  cols 0..W-1   (i-1, j-1) (i, j-1) (i+1, j-1)   (the case of Alg. 1)
 *     R2L  cols W-1..0   (i-1, j+1) (i, j+1) (i+1, j+1)
 *
 *   The backward (Alg. 2) is the exact adjoint for the loss <dy, y>.
 *
 *   Local GSPN (Sec. 4.1 "Local vs Global GSPN"; App. "CUDA Implementation",
 *   Alg. 1's groups of kNItems lines): `group_h` > 0 splits the rows into
 *   groups of group_h consecutive rows, [k*group_h, (k+1)*group_h) (the last
 *   group may be shorter); T2B and B2T restart from a zero state at the first
 *   row they visit in each group.  `group_w` does the same for the columns
 *   and L2R / R2L.  0 (or a value >= the line count) is the global scan.
 *
 *   Weight normalisation (Sec. 3.3, Eq. 6), flag GSPN_FLAG_W_LOGITS: w holds
 *   logits l and the scan uses w_k = sigmoid(l_k) / sum_k' sigmoid(l_k'), the
 *   sum over the three neighbours, or with GSPN_FLAG_EDGE_RENORM over the
 *   neighbours that lie on the line (the m_i non-zero entries of row i);
 *   dw is then the gradient with respect to the logits.
 *
 * Layouts (all tensors contiguous, element type `dtype`):
 *   x, lam, u, y, dy, dx, dlam, du : (B, C, H, W)
 *   w, dw                          : (n, 3, B, C, H, W), n = popcount(mask), the
 *                                    directions in increasing bit order; w[d][k] is
 *                                    the weight the RECEIVING pixel gives its
 *                                    neighbour k, stored at that pixel's (i, j).
 *   lam and u are shared by all directions, and y merges them, unless a
 *   per-direction flag is set (see GSPN_FLAG_*): then that tensor (and its
 *   gradient) is (n, B, C, H, W), one map per direction in the same order as
 *   w, and with GSPN_FLAG_Y_PER_DIR y_d = u_d * h_d is returned unmerged.
 *
 * Arithmetic: inputs are widened to fp32, every sum and product is fp32, and
 * each output element is rounded once (round-to-nearest-even for bf16).
 *
 * Ownership: every data pointer is device memory owned by the caller.  The
 * library allocates nothing; scratch memory is passed in as `workspace`
 * (size from the matching *_workspace_bytes call, 256-byte aligned).  No state
 * is kept between calls, so calls on different streams are independent.
 *
 * Empty problems: if B, C, H or W is 0 there is nothing to compute; the call
 * returns GSPN_OK after checking dtype, mask and algo, and pointers are not
 * inspected.
 *
 * Errors: 0 on success, a positive GSPN_ERR_* otherwise.  Arguments are
 * checked on the host before anything is launched; on an error nothing is
 * written.  Launch failures return GSPN_ERR_HIP.  Kernels run asynchronously
 * on `stream` (a hipStream_t; NULL = the default stream), so a device fault
 * surfaces at the caller's next synchronisation.
 */
#ifndef GSPN_H
#define GSPN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { GSPN_F32 = 0, GSPN_BF16 = 1 } gspn_dtype;

/* Options of a scan call (the `flags` argument, OR-ed together). */
enum {
  GSPN_FLAG_W_LOGITS = 1u,    /* w holds logits, normalised by Eq. 6 inside the call */
  GSPN_FLAG_EDGE_RENORM = 2u, /* with W_LOGITS: normalise over the on-line neighbours only */
  GSPN_FLAG_LAM_PER_DIR = 4u, /* lam and dlam are (n, B, C, H, W) */
  GSPN_FLAG_U_PER_DIR = 8u,   /* u and du are (n, B, C, H, W) */
  GSPN_FLAG_Y_PER_DIR = 16u,  /* y and dy are (n, B, C, H, W): y_d = u_d * h_d, not merged */
  GSPN_FLAG_SAVE_STATE = 32u  /* keep the forward's states for the backward (Alg. 2 takes the
                                 forward's H as an input): see below */
};

/* GSPN_FLAG_SAVE_STATE.  Forward: the call also leaves every direction's h and
 * sum_d h_d (fp32) at the start of its workspace.  Backward (same inputs,
 * shape, mask, groups, flags and algo): the call reads them there instead of
 * recomputing the forward scan.  The backward's workspace must therefore begin
 * with the bytes the forward left: size one buffer with
 * gspn_scan_bwd_workspace_bytes(..., flags) (which covers the forward's size)
 * and pass it to both calls, without touching the inputs in between.  dx, dw
 * and dlam are the same bits as without the flag; du adds the directions in
 * the forward's order.  Taken by the two-pass family with merged outputs and
 * a horizontal direction in the mask (the families that keep a plane on chip
 * recompute there at no HBM cost): the forward then returns GSPN_ERR_ALIGN for
 * tensors that are not 16-byte aligned instead of falling back to streaming.
 * For every other problem the flag changes nothing.  gspn_scan_fwd_noalloc
 * refuses it. */

enum {
  GSPN_DIR_T2B = 1u, /* top to bottom */
  GSPN_DIR_B2T = 2u, /* bottom to top */
  GSPN_DIR_L2R = 4u, /* left to right */
  GSPN_DIR_R2L = 8u  /* right to left */
};

enum {
  GSPN_OK = 0,
  GSPN_ERR_NULL = 1,        /* a required pointer is NULL */
  GSPN_ERR_SHAPE = 2,       /* a dimension < 0, or an element count overflows int64 */
  GSPN_ERR_MASK = 3,        /* mask is 0 or has bits above bit 3 */
  GSPN_ERR_DTYPE = 4,       /* unknown dtype */
  GSPN_ERR_ALIGN = 5,       /* a pointer is not aligned to its element size (workspace: 256 B) */
  GSPN_ERR_ALIAS = 6,       /* an output overlaps an input or another output */
  GSPN_ERR_UNSUPPORTED = 7, /* H or W above GSPN_MAX_LINE, unknown flags, EDGE_RENORM without
                               W_LOGITS, a negative group, or a forced algorithm that cannot run */
  GSPN_ERR_WORKSPACE = 8,   /* workspace NULL or smaller than required */
  GSPN_ERR_HIP = 9          /* a HIP launch or runtime call failed */
};

/* Longest line (H and W) the kernels accept. */
#define GSPN_MAX_LINE 4096

/* Algorithm selection (the `algo` argument).  AUTO picks the fastest kernel
 * family for the shape, groups and flags; the others force one family (for
 * testing), and return GSPN_ERR_UNSUPPORTED when it cannot take the problem.
 * Every family takes groups, GSPN_FLAG_W_LOGITS and GSPN_FLAG_EDGE_RENORM.
 * The per-direction flags are taken by the streaming family, by the resident
 * family's generic forward (unmerged y, per-direction lam, and per-direction
 * u with unmerged y) and by its per-wave backward (square planes of 16, 28,
 * 32, 56 or 64); GSPN_FLAG_Y_PER_DIR alone also by the two-pass family.  AUTO
 * picks among those. */
enum {
  GSPN_ALGO_AUTO = 0,
  GSPN_ALGO_RESIDENT = 1, /* whole plane kept on chip, all directions in one kernel */
  GSPN_ALGO_STREAM = 2,   /* one pass per direction through an fp32 workspace */
  GSPN_ALGO_RESIDENT_GENERIC = 3, /* resident family without size-specialised kernels */
  GSPN_ALGO_TWO_PASS = 4 /* for planes too large to keep on chip.  Forward: the
                            vertical directions in one pass, the horizontal pair in
                            blocks of 128-byte columns, partial sums in an fp32
                            workspace (two B*C*H*W arrays when both vertical
                            directions and a horizontal one are in the mask, one
                            otherwise).  Backward (a horizontal direction in the
                            mask): each horizontal direction recomputes its h into
                            the workspace block by block, then runs the adjoint over
                            the blocks in reverse order; the vertical directions
                            recompute their h in one pass and run both adjoints in
                            another.  Workspace: three fp32 B*C*H*W arrays (four
                            with both vertical directions) and 6*B*C*H floats.
                            Unmerged outputs (GSPN_FLAG_Y_PER_DIR): the forward
                            writes each direction's y and needs only the column
                            state; the backward seeds each direction from its dy.
                            GSPN_FLAG_SAVE_STATE: the forward keeps every h and
                            the sum (one fp32 array per direction, one for the
                            sum, and the column state), the backward runs only
                            the adjoints on them (see the flag).
                            Needs W * element size a multiple of 16 bytes and at
                            least 128 bytes, W <= 4096 (bf16) or 2048 (f32), and
                            16-byte aligned tensors (AUTO falls back to streaming). */
};

/* Bytes of workspace gspn_scan_fwd needs for this problem (0 if none). */
size_t gspn_scan_fwd_workspace_bytes(int64_t B, int64_t C, int64_t H, int64_t W, uint32_t mask,
                                     gspn_dtype dtype, int64_t group_h, int64_t group_w,
                                     uint32_t flags, int algo);

/*
 * Forward scan (Eq. 1-2): y = u * sum_{d in mask} h_d.
 *   x, w, lam, u : inputs (see layouts above); y : output, fully overwritten.
 *   group_h, group_w : local-GSPN group lengths (0 = global), see above.
 *   flags        : GSPN_FLAG_* options (0 = plain weights, shared lam/u, merged y).
 *   workspace    : device scratch of at least gspn_scan_fwd_workspace_bytes()
 *                  bytes, may be NULL when that size is 0.
 */
int gspn_scan_fwd(const void* x, const void* w, const void* lam, const void* u, void* y,
                  int64_t B, int64_t C, int64_t H, int64_t W, uint32_t mask, gspn_dtype dtype,
                  int64_t group_h, int64_t group_w, uint32_t flags, int algo,
                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * Forward scan that allocates nothing and takes no workspace, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation).  Same arguments and result as
 * gspn_scan_fwd with GSPN_ALGO_AUTO; the scratch memory the kernel families
 * need comes from a fixed array of GSPN_NOALLOC_SCRATCH_BYTES inside the
 * library, one per GPU, held until the process ends.
 *   Returns GSPN_ERR_WORKSPACE, before anything runs, when the problem needs
 *   more scratch than that (gspn_scan_fwd_workspace_bytes(..., AUTO) tells).
 *   Every call on one GPU shares that GPU's array: calls that overlap in time
 *   on one GPU (different streams, or host threads) race and must not be
 *   issued.  Nothing in the array needs to start at zero; it keeps the last
 *   call's contents.
 */
#define GSPN_NOALLOC_SCRATCH_BYTES (64u << 20)
int gspn_scan_fwd_noalloc(const void* x, const void* w, const void* lam, const void* u, void* y,
                          int64_t B, int64_t C, int64_t H, int64_t W, uint32_t mask,
                          gspn_dtype dtype, int64_t group_h, int64_t group_w, uint32_t flags,
                          void* stream);

/* Bytes of workspace gspn_scan_bwd needs for this problem (0 if none).  With
 * GSPN_ALGO_AUTO the size covers every pointer alignment: AUTO runs the
 * streaming family, which needs a workspace (never more than the two-pass
 * one), when a tensor the resident or two-pass kernels would read or write as
 * 16-byte vectors is only element-aligned. */
size_t gspn_scan_bwd_workspace_bytes(int64_t B, int64_t C, int64_t H, int64_t W, uint32_t mask,
                                     gspn_dtype dtype, int64_t group_h, int64_t group_w,
                                     uint32_t flags, int algo);

/*
 * Backward scan (Alg. 2, exact adjoint of Eq. 1-2) for the loss <dy, y>:
 *   inputs dy, x, w, lam, u (same values, groups and flags as the forward call);
 *   outputs dx, dlam, du and dw (shaped like x, lam, u and w), fully
 *   overwritten (not accumulated).  With GSPN_FLAG_W_LOGITS dw is the
 *   gradient with respect to the logits.  The forward state is recomputed
 *   inside, so no tensor from the forward call is needed (with
 *   GSPN_FLAG_SAVE_STATE the two-pass family reads the state the forward
 *   left at the start of the workspace instead).
 */
int gspn_scan_bwd(const void* dy, const void* x, const void* w, const void* lam, const void* u,
                  void* dx, void* dw, void* dlam, void* du,
                  int64_t B, int64_t C, int64_t H, int64_t W, uint32_t mask, gspn_dtype dtype,
                  int64_t group_h, int64_t group_w, uint32_t flags, int algo,
                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * Plain device-to-device copy of `bytes` bytes (src and dst 16-byte aligned,
 * not overlapping).  Not part of the scan: it is the reference kernel of known
 * traffic (reads `bytes`, writes `bytes`) against which hardware byte counters
 * (rocprofv3 FETCH_SIZE / WRITE_SIZE) of the scan kernels are scaled.
 * Asynchronous on `stream`.
 */
int gspn_copy_calibration(const void* src, void* dst, size_t bytes, void* stream);

/* Static, NUL-terminated description of a status code. */
const char* gspn_strerror(int status);

/* Library version as 10000*major + 100*minor + patch. */
int gspn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* GSPN_H */
