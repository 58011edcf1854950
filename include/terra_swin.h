/*
 * terra_swin.h - C ABI of the MI355X (gfx950) shifted-window attention path.
 *
 * The library implements the per-GPU hot path inside the Swin blocks of the
 * paper's hierarchical Earth-forecasting model: the token route between the
 * spatially contiguous layout and the window-major layout (Sec. IV-D), and
 * shifted-window multi-head self-attention with relative-position bias,
 * forward and backward (W-MSA / SW-MSA of the Swin blocks, Sec. IV-A).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Geometry.  The Transformer-stage token grid is H x W (Sec. IV-D, Eq. (2)),
 *   B images, C = heads * head_dim channels (Table I: d, N_h), attention
 *   window wh x ww (Table I: w, generalised to a rectangle) and window shift
 *   (sh, sw) with 0 <= sh < wh <= H, 0 <= sw < ww <= W.
 * Shift.  The grid is rolled so that content moves toward the top-left: the
 *   rolled coordinate of original token (u, v) is ((u - sh) mod H,
 *   (v - sw) mod W).  Windows partition the rolled grid (Eq. (2)); when wh
 *   does not divide H (ww does not divide W) the last window row (column) is
 *   partial - there is no padding.
 * Mask.  mask_flags bit 0 (TERRA_MASK_LAT) labels the sh rows that wrapped
 *   across the latitude edge, bit 1 (TERRA_MASK_LON) the sw wrapped columns;
 *   tokens attend only to tokens of their own window with equal labels.
 *   Longitude is normally periodic (bit 1 clear).
 * Layouts.  NHWC tensors are B x H x W x C, contiguous.  Window-major tensors
 *   are B x (H*W) x C: per image, windows in row-major order (Sec. V-A,
 *   Eq. (4) flattening), tokens row-major over each window's actual extent,
 *   channel c = h * head_dim + e.  LSE is B x heads x (H*W) float32 in
 *   window-major token order.  Bias tables are float32
 *   [2wh-1][2ww-1][heads]; the bias of query q and key k is
 *   T[a_q - a_k + wh - 1][c_q - c_k + ww - 1][h], (a, c) = in-window offset.
 * Element types.  TERRA_F32 (float), TERRA_BF16 (bfloat16 storage, float32
 *   accumulation, results rounded to nearest even) or TERRA_F16 (IEEE half
 *   storage, the paper's training precision, float32 accumulation).  Bias
 *   tables, LSE and the bias-table gradient are always float32.
 * Memory.  Every tensor pointer is a DEVICE pointer allocated by the caller;
 *   the library allocates nothing and keeps no device state.  Geometry
 *   structs and host arrays stay owned by the caller.  Tensors of one call
 *   must not overlap unless stated.
 * Streams.  `stream` is a hipStream_t (NULL = the default stream).  Calls
 *   only enqueue work on it and never synchronise.
 * Errors.  Every int-returning call returns a terra_status.  Argument checks
 *   run on the host before any device work, so an error status means nothing
 *   was enqueued (except TERRA_ERR_HIP, reported by the HIP runtime after a
 *   launch).  terra_last_error() gives a message for the calling thread.
 */
#ifndef TERRA_SWIN_H
#define TERRA_SWIN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct terra_geom {
  int32_t B, H, W, C;        /* images, grid rows/cols, channels          */
  int32_t heads, head_dim;   /* C == heads * head_dim                     */
  int32_t wh, ww;            /* window extent                             */
  int32_t sh, sw;            /* window shift                              */
  int32_t mask_flags;        /* TERRA_MASK_LAT | TERRA_MASK_LON           */
} terra_geom;

enum terra_dtype { TERRA_F32 = 0, TERRA_BF16 = 1, TERRA_F16 = 2 };

enum terra_status {
  TERRA_OK = 0,
  TERRA_ERR_INVALID = 1,      /* geometry rule broken, null pointer, bad dtype value */
  TERRA_ERR_UNSUPPORTED = 2,  /* valid but outside what the kernels handle          */
  TERRA_ERR_WORKSPACE = 3,    /* workspace missing or smaller than required         */
  TERRA_ERR_HIP = 4           /* the HIP runtime reported an error                  */
};

#define TERRA_MASK_LAT 1
#define TERRA_MASK_LON 2

/* Library version, major*10000 + minor*100 + patch. */
int terra_version(void);

/* Checks the geometry rules above (host only, no device call).  Returns
 * TERRA_OK, TERRA_ERR_INVALID, or TERRA_ERR_UNSUPPORTED when the attention
 * kernels cannot take it (head_dim not 32, 64 or 128, more than 8192 bias
 * bins per head, more than 2^31 elements per tensor).  Routing accepts any
 * geometry that is valid. */
int terra_validate_geometry(const terra_geom* g);

/* Window grid size Mh = ceil(H/wh), Mw = ceil(W/ww) (Eq. (2), with ragged
 * edges).  Host pointers. */
int terra_window_count(const terra_geom* g, int32_t* Mh, int32_t* Mw);

/* Window-major layout of ONE image (Sec. IV-D / Sec. V-A): for window
 * w = i*Mw + j, offsets[w] is its first token slot and counts[w] its token
 * count rows_i * cols_j; offsets[Mh*Mw] = H*W.  Host arrays of Mh*Mw+1 and
 * Mh*Mw int32 entries owned by the caller.  Image b's slots start at b*H*W. */
int terra_window_layout(const terra_geom* g, int32_t* offsets, int32_t* counts);

/* Token route, NHWC -> window-major (Sec. IV-D: the route gathers every
 * token into its window-major slot after the window shift).  Bit copy of
 * B*H*W*C elements of `dtype`; x_nhwc and y_win must not overlap.
 * d_offsets / d_counts (nullable DEVICE int32 arrays of Mh*Mw+1 and Mh*Mw
 * entries) receive the per-window first slots and valid-token counts of one
 * image, as terra_window_layout gives them on the host, written on the same
 * stream. */
int terra_window_route(const terra_geom* g, int dtype, const void* x_nhwc,
                       void* y_win, int32_t* d_offsets, int32_t* d_counts,
                       void* stream);

/* Inverse token route, window-major -> NHWC: the exact inverse scatter of
 * terra_window_route, and also its adjoint (the backward of the route is the
 * inverse route, Sec. IV-D). */
int terra_window_unroute(const terra_geom* g, int dtype, const void* y_win,
                         void* x_nhwc, void* stream);

/* Shifted-window attention forward (Sec. IV-A, W-MSA / SW-MSA).  For every
 * image, window and head: S = Q K^T / sqrt(head_dim) + bias, masked pairs
 * excluded, P = softmax(S), O = P V, LSE = ln sum exp S (natural log).
 * q, k, v, o: window-major, `dtype`; bias_table: float32 table;
 * lse: float32 B x heads x (H*W).  o and lse are overwritten.
 * o_lo (nullable, same shape and type as o): where
 * terra_winattn_uses_o_lo(g, dtype) is 1, the forward forms O with P
 * entering the P V product as two 16-bit parts (so that the float32 O is
 * exact to about 16 significant bits) and writes O - round(O), rounded to
 * `dtype`, into o_lo.  Passed on to the backward, it gives
 * D_q = <dO_q, O_q> without an extra sweep over the keys.  Elsewhere o_lo
 * is neither written nor read, and with o_lo NULL the forward is unchanged. */
int terra_winattn_fwd(const terra_geom* g, int dtype, const void* q,
                      const void* k, const void* v, const float* bias_table,
                      void* o, void* o_lo, float* lse, void* stream);

/* 1 when the forward writes o_lo and the backward reads it for this
 * geometry and element type (float16 and bfloat16 with windows of more
 * than 256 tokens, where the key sweep it replaces costs more than the
 * split product and the extra traffic), 0 when o_lo is ignored, -status on
 * invalid input. */
int terra_winattn_uses_o_lo(const terra_geom* g, int dtype);

/* Bytes of device workspace terra_winattn_bwd (and terra_winattn_bwd_nhwc)
 * needs for this geometry (0 on invalid input). */
size_t terra_winattn_bwd_workspace_bytes(const terra_geom* g, int dtype);

/* Shifted-window attention backward.  Inputs are the forward's inputs, its
 * outputs o, o_lo and lse, and the upstream gradient dout (window-major).
 * Outputs dq, dk, dv (window-major, `dtype`) and dbias_table (float32,
 * table shape, summed over images, windows and allowed pairs) are
 * OVERWRITTEN.  dS = P * (dP - D), D_q = sum_k P[q,k] dP[q,k] = <dO_q, O_q>
 * for the exact O, in float32: from o + o_lo when o_lo is not NULL and
 * terra_winattn_uses_o_lo(g, dtype) is 1, otherwise recomputed inside each
 * window from P and dP.  The rounded O alone is not used for it: D's
 * rounding error, alike for every key of a query, would add up over the
 * windows in the bias-table gradient.  The bias-table gradient is reduced
 * in a fixed order, so results are bit-reproducible.
 * workspace: device buffer of at least terra_winattn_bwd_workspace_bytes. */
int terra_winattn_bwd(const terra_geom* g, int dtype, const void* q,
                      const void* k, const void* v, const void* o,
                      const void* o_lo, const void* dout, const float* lse,
                      const float* bias_table, void* dq, void* dk, void* dv,
                      float* dbias_table, void* workspace,
                      size_t workspace_bytes, void* stream);

/* Fused route + attention forward: the same computation as
 * terra_winattn_fwd with q, k, v and o as NHWC tensors read and written in
 * place (Sec. IV-D route and its inverse folded into the kernels: row t of
 * window (i, j) is read from, and its output written to, the grid point
 * ((i*wh + t/cols + sh) mod H, (j*ww + t%cols + sw) mod W)).  lse is
 * float32 B x heads x (H*W) in NHWC token order (index u*W + v).  Results
 * equal terra_window_unroute of the window-major call's results, bit for
 * bit. */
int terra_winattn_fwd_nhwc(const terra_geom* g, int dtype, const void* q,
                           const void* k, const void* v,
                           const float* bias_table, void* o, void* o_lo,
                           float* lse, void* stream);

/* Fused route + attention backward: terra_winattn_bwd with q, k, v, o,
 * o_lo, dout, dq, dk, dv as NHWC tensors and lse in NHWC token order, as written
 * by terra_winattn_fwd_nhwc.  Needs the workspace of
 * terra_winattn_bwd_workspace_bytes (the same size for both layouts). */
int terra_winattn_bwd_nhwc(const terra_geom* g, int dtype, const void* q,
                           const void* k, const void* v, const void* o,
                           const void* o_lo, const void* dout, const float* lse,
                           const float* bias_table, void* dq, void* dk,
                           void* dv, float* dbias_table, void* workspace,
                           size_t workspace_bytes, void* stream);

/* Allocation-free fused backward, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): terra_winattn_bwd_nhwc with its workspace taken from a
 * device array the library holds, TERRA_SCRATCH_BYTES per GPU, kept until
 * the process ends.  The caller still passes every input and output.  The
 * call allocates nothing (its first call on a device looks up that device's
 * array address once).  Geometries whose workspace
 * (terra_winattn_bwd_workspace_bytes) exceeds TERRA_SCRATCH_BYTES return
 * TERRA_ERR_UNSUPPORTED before any device work.  Every call on one GPU
 * shares that GPU's array: calls that overlap on one GPU (concurrent
 * streams, threads) race and must be ordered by the caller.  No part of the
 * array needs to start at zero: each call writes everything it reads. */
#define TERRA_SCRATCH_BYTES (32u << 20)
int terra_winattn_bwd_nhwc_noalloc(const terra_geom* g, int dtype, const void* q,
                                   const void* k, const void* v, const void* o,
                                   const void* o_lo, const void* dout,
                                   const float* lse,
                                   const float* bias_table, void* dq, void* dk,
                                   void* dv, float* dbias_table, void* stream);

/* ---------------------------------------------------------------------------
 * One Swin block around the attention (Sec. IV-A Swin blocks, whose linear
 * layers TP shards in Sec. IV-C; widths as in Table III), pre-norm with two
 * residual branches, on NHWC tokens of width C = d:
 *   x1 = x  + Proj(A(LN1(x) W_qkv^T + b_qkv)),  Proj(o) = o W_proj^T + b_proj
 *   x2 = x1 + GELU(LN2(x1) W_fc1^T + b_fc1) W_fc2^T + b_fc2
 * LN over the C channels of a token (biased variance, eps 1e-5, gain and
 * shift); GELU the exact (erf) form; A the shifted-window attention of
 * terra_winattn_fwd_nhwc with the bias table.  W_qkv is 3C x C (rows
 * [0,C) -> Q, [C,2C) -> K, [2C,3C) -> V), W_proj C x C, W_fc1 4C x C,
 * W_fc2 C x 4C, all row-major (out x in) bf16; gains, shifts and biases
 * float32.  Element type TERRA_BF16 only; C must be a multiple of 128 and
 * at most 2048, and the geometry must suit the attention.
 * LayerNorm never writes its output to memory: the forward folds it into
 * the projection that follows it, the backward applies it to the staged
 * operand of the weight gradient; Q, K and V are written straight as the
 * NHWC tensors the fused attention reads.
 * ------------------------------------------------------------------------- */

typedef struct terra_block_params {      /* device pointers                 */
  const float *ln1_g, *ln1_b;            /* C                               */
  const void* w_qkv;                     /* bf16 3C x C                     */
  const float* b_qkv;                    /* 3C                              */
  const void* w_proj;                    /* bf16 C x C                      */
  const float* b_proj;                   /* C                               */
  const float *ln2_g, *ln2_b;            /* C                               */
  const void* w_fc1;                     /* bf16 4C x C                     */
  const float* b_fc1;                    /* 4C                              */
  const void* w_fc2;                     /* bf16 C x 4C                     */
  const float* b_fc2;                    /* C                               */
} terra_block_params;

typedef struct terra_block_grads {       /* float32 device outputs, same shapes as the parameters */
  float *ln1_g, *ln1_b, *w_qkv, *b_qkv, *w_proj, *b_proj, *ln2_g, *ln2_b, *w_fc1, *b_fc1, *w_fc2, *b_fc2;
} terra_block_grads;

/* Activations the forward writes and the backward reads (device, caller
 * owned; T = B*H*W tokens): LN statistics (float32 T each), Q, K, V and the
 * attention output O (bf16 NHWC, T x C), the attention LSE (float32
 * B x heads x H*W, NHWC token order), x1 (bf16 T x C), the MLP
 * pre-activation h and its GELU a (bf16 T x 4C). */
typedef struct terra_block_saved {
  float *mu1, *rstd1, *mu2, *rstd2;
  void *q, *k, *v, *o;
  float* lse;
  void* x1;
  void *h, *a;
} terra_block_saved;

/* Device workspace terra_block_fwd needs (0 on invalid input): the QKV and
 * first MLP weights with the LayerNorm gains folded in, and two per-output
 * vectors each. */
size_t terra_block_fwd_workspace_bytes(const terra_geom* g, int dtype);

/* Forward: x (bf16 NHWC) -> x2 (bf16 NHWC), filling `saved`.  Each
 * LayerNorm is folded into the projection after it: with
 * Wf[n][k] = bf16(W[n][k] gain_k), s_n = sum_k Wf[n][k] and
 * c_n = b_n + sum_k W[n][k] shift_k, LN(z) W^T + b = rstd (z Wf^T - mean s) + c,
 * so the matrix cores run on the raw activations and the normalisation is
 * applied to the accumulators. */
int terra_block_fwd(const terra_geom* g, int dtype, const void* x, const terra_block_params* p,
                    const float* bias_table, void* x2, const terra_block_saved* saved, void* workspace,
                    size_t workspace_bytes, void* stream);

/* Device workspace terra_block_bwd needs (0 on invalid input). */
size_t terra_block_bwd_workspace_bytes(const terra_geom* g, int dtype);

/* Backward from the upstream gradient dx2: dx (bf16 NHWC), every parameter
 * gradient (float32, summed over all tokens, overwritten) and the bias-table
 * gradient (overwritten).  x and `saved` as left by terra_block_fwd.
 * Reductions over tokens run in a fixed order (bit-reproducible). */
int terra_block_bwd(const terra_geom* g, int dtype, const void* dx2, const void* x,
                    const terra_block_params* p, const float* bias_table,
                    const terra_block_saved* saved, void* dx, const terra_block_grads* grads,
                    float* dbias_table, void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Window assignment across ranks and the per-rank token route.
 *
 * On a multi-GPU run the token grid is held in DMP height stripes (the I/O
 * topology, Sec. IV-B) and attention runs on complete windows owned by WP
 * ranks (Sec. IV-C).  The calls below plan the ragged row-major ownership of
 * Sec. V-A (Eq. (4)), list for one rank the rectangles of the grid it must
 * receive from other ranks for its route (the boundary fragments of the
 * shift route, Sec. IV-D), and run that rank's route and its inverse from
 * its own stripe plus a buffer holding those fragments.  On one GPU the
 * ranks are run one after another, and the fragment copy stands in for the
 * point-to-point exchange.
 *
 * Stripes.  Rank r of P holds grid rows [floor(r H / P), floor((r+1) H / P))
 *   of every image, as a B x rows x W x C tensor (the floor rule of Eq. (4)
 *   applied to rows; equal stripes when P divides H, as on the paper's
 *   padded grids).
 * Windows.  Rank r owns windows [L_r, R_r), L_r = floor(r M / P), of every
 *   image, M = Mh * Mw in row-major order (Eq. (4)); its window-major
 *   tensor is B x (slot_end - slot_begin) x C, the slots of those windows in
 *   the layout of terra_window_route.
 * Fragments.  Rows [u0, u1) x columns [v0, v1) of the original grid held by
 *   rank src_rank, stored row-major from token `offset` of the receiving
 *   rank's fragment buffer (B x frag_tokens x C, image-major).  They are
 *   sorted by source rank, so everything one rank sends to another is one
 *   contiguous run of the buffer.
 * ------------------------------------------------------------------------- */

#define TERRA_MAX_FRAGMENTS 64

typedef struct terra_rank_plan {
  int32_t win_begin, win_end;     /* Eq. (4) window range [L_r, R_r)          */
  int32_t slot_begin, slot_end;   /* its window-major slots, per image        */
  int32_t row_begin, row_end;     /* DMP stripe rows held by the rank         */
  int32_t nfrag;                  /* fragments received from other ranks      */
  int32_t frag_tokens;            /* tokens per image in the fragment buffer  */
} terra_rank_plan;

typedef struct terra_fragment {
  int32_t src_rank;               /* rank whose stripe holds the rectangle    */
  int32_t u0, u1, v0, v1;         /* grid rows [u0, u1), columns [v0, v1)     */
  int32_t offset;                 /* first token in the fragment buffer       */
} terra_fragment;

/* Eq. (3): padded input size of the fixed window assignment on an m x n WP
 * mesh, Hhat = ceil(H / (p alpha w m)) p alpha w m (What likewise with n),
 * for patch size p, down-sampling stride alpha and window w.  m = n = 1
 * gives the least padding to whole windows.  overhead (nullable) receives
 * Hhat What / (H W) - 1.  Host only. */
int terra_plan_padded_grid(int32_t H, int32_t W, int32_t p, int32_t alpha, int32_t w, int32_t m,
                           int32_t n, int32_t* Hhat, int32_t* What, double* overhead);

/* Eq. (4): bounds[r] = floor(r M / ranks) for r = 0 .. ranks (ranks + 1
 * host entries); rank r owns windows [bounds[r], bounds[r+1]).  Host only. */
int terra_plan_window_ranges(int64_t M, int32_t ranks, int64_t* bounds);

/* Plan of rank `rank` among `ranks` for the geometry g (its window range,
 * slots, stripe and received fragments).  frags (nullable) receives
 * plan->nfrag entries, at most TERRA_MAX_FRAGMENTS.  TERRA_ERR_UNSUPPORTED
 * when the rank would receive more fragments (stripes far thinner than a
 * window).  Host only. */
int terra_plan_rank(const terra_geom* g, int32_t ranks, int32_t rank, terra_rank_plan* plan,
                    terra_fragment* frags);

/* Route of one rank: its window-major tensor y_win (B x (slot_end -
 * slot_begin) x C) gathered from its stripe and its fragment buffer
 * (layouts above).  Equals the corresponding slots of terra_window_route of
 * the whole grid, bit for bit.  Device pointers; frag_buf may be NULL when
 * the plan has no fragments. */
int terra_window_route_rank(const terra_geom* g, int dtype, int32_t ranks, int32_t rank,
                            const void* stripe, const void* frag_buf, void* y_win, void* stream);

/* Inverse of terra_window_route_rank (its backward, Sec. IV-D): scatters
 * y_win back to the rank's stripe and its fragment buffer.  Every element
 * of the stripe that the rank's windows cover, and every fragment token, is
 * overwritten; the rest is left as it was. */
int terra_window_unroute_rank(const terra_geom* g, int dtype, int32_t ranks, int32_t rank,
                              const void* y_win, void* stripe, void* frag_buf, void* stream);

/* The exchange of the fragments of rank dst_rank's plan whose source is
 * src_rank: pack copies them from src_rank's stripe into dst_rank's
 * fragment buffer (the send and the receive of the point-to-point exchange
 * in one copy), unpack copies them back (the backward).  Nothing is done
 * when dst_rank receives nothing from src_rank. */
int terra_fragment_pack(const terra_geom* g, int dtype, int32_t ranks, int32_t dst_rank,
                        int32_t src_rank, const void* src_stripe, void* frag_buf, void* stream);
int terra_fragment_unpack(const terra_geom* g, int dtype, int32_t ranks, int32_t dst_rank,
                          int32_t src_rank, const void* frag_buf, void* src_stripe, void* stream);

/* Static string naming a status code. */
const char* terra_status_string(int status);

/* Message of the last failed call on the calling thread ("" if none). */
const char* terra_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TERRA_SWIN_H */
