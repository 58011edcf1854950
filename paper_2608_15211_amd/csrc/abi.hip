// abi.hip - C ABI of the shifted-window attention library (declared in
// include/terra_swin.h): host-side argument checks, geometry set-up and
// dispatch to the gfx950 kernels.  No allocation, no synchronisation.
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <initializer_list>
#include <mutex>
#include <string>

#include "terra_common.h"
#include "terra_plan.h"
#include "terra_block.h"
#include "../../include/terra_swin.h"

namespace terra {
hipError_t launch_route(const Geo& g, int row_bytes, const void* src, void* dst, bool forward,
                        hipStream_t stream);
hipError_t launch_layout(const Geo& g, int32_t* offsets, int32_t* counts, hipStream_t stream);
hipError_t launch_block_fwd(const Geo& g, const void* x, const BlockParams& p, const float* table, void* x2,
                            const BlockSaved& s, void* ws, hipStream_t st);
size_t block_fwd_workspace(const Geo& g);
hipError_t launch_block_bwd(const Geo& g, const void* dx2, const void* x, const BlockParams& p, const float* table,
                            const BlockSaved& s, void* dx, const BlockGrads& gr, float* dtable, void* ws,
                            hipStream_t st);
size_t block_bwd_workspace(const Geo& g);
hipError_t launch_attn_fwd(const Geo& g, int dt, bool nhwc, const void* q, const void* k,
                           const void* v, const float* table, void* o, void* olo, float* lse,
                           hipStream_t st);
hipError_t launch_attn_bwd(const Geo& g, int dt, bool nhwc, const void* q, const void* k,
                           const void* v, const void* o, const void* olo, const void* dout,
                           const float* lse, const float* table, void* dq, void* dk, void* dv,
                           float* dtab, void* ws, hipStream_t st);
bool attn_uses_olo(const Geo& g, int dt);
size_t bwd_workspace(const Geo& g, int dt);
size_t attn_max_lds(const Geo& g, int dt);
hipError_t launch_route_rank(const Geo& g, int row_bytes, const RankPlan& plan, const Frag* frags,
                             void* stripe, void* fbuf, void* y, bool forward, hipStream_t st);
hipError_t launch_frag_copy(const Geo& g, int row_bytes, const RankPlan& plan, const Frag* frags,
                            int src, int src_row_begin, int src_row_end, void* stripe, void* fbuf,
                            bool pack, hipStream_t st);
}  // namespace terra

namespace {

thread_local std::string g_last_error;

int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

int ok() {
  g_last_error.clear();
  return TERRA_OK;
}

int hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(TERRA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

constexpr int64_t kMaxElems = (int64_t)1 << 31;   // per tensor, attention kernels
constexpr int kMaxBins = 8192;                    // bias bins per head
constexpr size_t kMaxLds = 160 * 1024;            // LDS per workgroup on gfx950

// Geometry rules shared by every entry point.
int check_geom(const terra_geom* g) {
  if (!g) return fail(TERRA_ERR_INVALID, "geometry pointer is NULL");
  if (g->B < 1 || g->H < 1 || g->W < 1 || g->C < 1 || g->heads < 1 || g->head_dim < 1)
    return fail(TERRA_ERR_INVALID, "B, H, W, C, heads and head_dim must be >= 1");
  if ((int64_t)g->heads * g->head_dim != g->C)
    return fail(TERRA_ERR_INVALID, "C (%d) != heads (%d) * head_dim (%d)", g->C, g->heads,
                g->head_dim);
  if (g->wh < 1 || g->wh > g->H || g->ww < 1 || g->ww > g->W)
    return fail(TERRA_ERR_INVALID, "window %dx%d must satisfy 1 <= wh <= H (%d), 1 <= ww <= W (%d)",
                g->wh, g->ww, g->H, g->W);
  if (g->sh < 0 || g->sh >= g->wh || g->sw < 0 || g->sw >= g->ww)
    return fail(TERRA_ERR_INVALID, "shift (%d,%d) must satisfy 0 <= sh < wh, 0 <= sw < ww", g->sh,
                g->sw);
  if (g->mask_flags < 0 || g->mask_flags > 3)
    return fail(TERRA_ERR_INVALID, "mask_flags %d has bits other than 0 and 1", g->mask_flags);
  if ((int64_t)g->B * g->H * g->W >= ((int64_t)1 << 31))
    return fail(TERRA_ERR_UNSUPPORTED, "B*H*W must be below 2^31 tokens");
  return ok();
}

int check_dtype(int dtype) {
  if (dtype != TERRA_F32 && dtype != TERRA_BF16 && dtype != TERRA_F16)
    return fail(TERRA_ERR_INVALID, "dtype %d is not TERRA_F32, TERRA_BF16 or TERRA_F16", dtype);
  return ok();
}

terra::Geo make_geo(const terra_geom* g) {
  terra::Geo G;
  G.B = g->B; G.H = g->H; G.W = g->W; G.C = g->C; G.heads = g->heads; G.hd = g->head_dim;
  G.wh = g->wh; G.ww = g->ww; G.sh = g->sh; G.sw = g->sw; G.flags = g->mask_flags;
  G.Mh = (g->H + g->wh - 1) / g->wh;
  G.Mw = (g->W + g->ww - 1) / g->ww;
  G.nwin = G.Mh * G.Mw;
  G.HW = g->H * g->W;
  G.bstride = 2 * g->ww - 1;
  G.nbins = (2 * g->wh - 1) * G.bstride;
  terra::set_table_stride(G);
  terra::set_col_recips(G);
  G.cus = terra::kMaxCus;
  return G;
}

// Compute units of the current device (asked once per device), clamped to
// [1, kMaxCus]; the launchers size their persistent grids from it.
std::mutex g_cus_mu;
int g_cus[64] = {};
int device_cus() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    (void)hipGetLastError();
    return 256;
  }
  std::lock_guard<std::mutex> lock(g_cus_mu);
  if (g_cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1) {
      (void)hipGetLastError();
      n = 256;
    }
    g_cus[dev] = n > terra::kMaxCus ? terra::kMaxCus : n;
  }
  return g_cus[dev];
}

terra::Geo launch_geo(const terra_geom* g) {
  terra::Geo G = make_geo(g);
  G.cus = device_cus();
  return G;
}

// Attention-specific limits.
int check_attn(const terra_geom* g, int dtype) {
  int s = check_geom(g);
  if (s) return s;
  if ((s = check_dtype(dtype))) return s;
  if (g->head_dim != 32 && g->head_dim != 64 && g->head_dim != 128)
    return fail(TERRA_ERR_UNSUPPORTED, "head_dim %d: the attention kernels take 32, 64 or 128",
                g->head_dim);
  if ((int64_t)g->B * g->H * g->W * g->C >= kMaxElems)
    return fail(TERRA_ERR_UNSUPPORTED, "tensors above 2^31 elements are not supported");
  terra::Geo G = make_geo(g);
  if (G.nbins > kMaxBins)
    return fail(TERRA_ERR_UNSUPPORTED, "(2wh-1)(2ww-1) = %d bias bins exceeds %d", G.nbins,
                kMaxBins);
  if (terra::attn_max_lds(G, dtype) > kMaxLds)
    return fail(TERRA_ERR_UNSUPPORTED, "window needs more LDS than one workgroup has");
  return ok();
}

}  // namespace

extern "C" {

int terra_version(void) { return 100; }

int terra_validate_geometry(const terra_geom* g) {
  int s = check_geom(g);
  if (s) return s;
  if (g->head_dim != 32 && g->head_dim != 64 && g->head_dim != 128)
    return fail(TERRA_ERR_UNSUPPORTED, "head_dim %d: the attention kernels take 32, 64 or 128",
                g->head_dim);
  terra::Geo G = make_geo(g);
  if (G.nbins > kMaxBins)
    return fail(TERRA_ERR_UNSUPPORTED, "(2wh-1)(2ww-1) = %d bias bins exceeds %d", G.nbins,
                kMaxBins);
  if ((int64_t)g->B * g->H * g->W * g->C >= kMaxElems)
    return fail(TERRA_ERR_UNSUPPORTED, "tensors above 2^31 elements are not supported");
  return ok();
}

int terra_window_count(const terra_geom* g, int32_t* Mh, int32_t* Mw) {
  int s = check_geom(g);
  if (s) return s;
  if (!Mh || !Mw) return fail(TERRA_ERR_INVALID, "output pointer is NULL");
  terra::Geo G = make_geo(g);
  *Mh = G.Mh;
  *Mw = G.Mw;
  return ok();
}

int terra_window_layout(const terra_geom* g, int32_t* offsets, int32_t* counts) {
  int s = check_geom(g);
  if (s) return s;
  if (!offsets || !counts) return fail(TERRA_ERR_INVALID, "output pointer is NULL");
  terra::Geo G = make_geo(g);
  for (int i = 0; i < G.Mh; ++i)
    for (int j = 0; j < G.Mw; ++j) {
      const int w = i * G.Mw + j;
      offsets[w] = terra::win_offset(G, i, j);
      counts[w] = terra::win_rows(G, i) * terra::win_cols(G, j);
    }
  offsets[G.nwin] = G.HW;
  return ok();
}

static int route_common(const terra_geom* g, int dtype, const void* src, void* dst, bool forward,
                        int32_t* d_offsets, int32_t* d_counts, void* stream) {
  int s = check_geom(g);
  if (s) return s;
  if ((s = check_dtype(dtype))) return s;
  if (!src || !dst) return fail(TERRA_ERR_INVALID, "tensor pointer is NULL");
  if (src == dst) return fail(TERRA_ERR_INVALID, "route source and destination must differ");
  const int esize = dtype == TERRA_F32 ? 4 : 2;
  const int64_t row_bytes = (int64_t)g->C * esize;
  // The per-window chunk index must stay below 2^22 (worst case 2-byte chunks).
  if ((int64_t)g->wh * g->ww * (row_bytes / 2) >= ((int64_t)1 << 22))
    return fail(TERRA_ERR_UNSUPPORTED, "window of %d tokens x %lld bytes is too large to route",
                g->wh * g->ww, (long long)row_bytes);
  terra::Geo G = make_geo(g);
  if (d_offsets || d_counts) {
    s = hip_status(terra::launch_layout(G, d_offsets, d_counts, (hipStream_t)stream),
                   "terra_window_route layout launch");
    if (s) return s;
  }
  return hip_status(terra::launch_route(G, (int)row_bytes, src, dst, forward, (hipStream_t)stream),
                    forward ? "terra_window_route launch" : "terra_window_unroute launch");
}

int terra_window_route(const terra_geom* g, int dtype, const void* x_nhwc, void* y_win,
                       int32_t* d_offsets, int32_t* d_counts, void* stream) {
  return route_common(g, dtype, x_nhwc, y_win, true, d_offsets, d_counts, stream);
}

int terra_window_unroute(const terra_geom* g, int dtype, const void* y_win, void* x_nhwc,
                         void* stream) {
  return route_common(g, dtype, y_win, x_nhwc, false, nullptr, nullptr, stream);
}

}  // extern "C"

static int attn_fwd_common(const terra_geom* g, int dtype, bool nhwc, const void* q, const void* k,
                           const void* v, const float* bias_table, void* o, void* o_lo, float* lse,
                           void* stream) {
  int s = check_attn(g, dtype);
  if (s) return s;
  if (!q || !k || !v || !bias_table || !o || !lse)
    return fail(TERRA_ERR_INVALID, "tensor pointer is NULL");
  terra::Geo G = launch_geo(g);
  return hip_status(terra::launch_attn_fwd(G, dtype, nhwc, q, k, v, bias_table, o, o_lo, lse,
                                           (hipStream_t)stream),
                    nhwc ? "terra_winattn_fwd_nhwc launch" : "terra_winattn_fwd launch");
}

static int attn_bwd_common(const terra_geom* g, int dtype, bool nhwc, const void* q, const void* k,
                           const void* v, const void* o, const void* o_lo, const void* dout,
                           const float* lse,
                           const float* bias_table, void* dq, void* dk, void* dv,
                           float* dbias_table, void* workspace, size_t workspace_bytes,
                           void* stream) {
  int s = check_attn(g, dtype);
  if (s) return s;
  if (!q || !k || !v || !o || !dout || !lse || !bias_table || !dq || !dk || !dv || !dbias_table)
    return fail(TERRA_ERR_INVALID, "tensor pointer is NULL");
  const size_t need = terra::bwd_workspace(make_geo(g), dtype);
  terra::Geo G = launch_geo(g);
  if (!workspace || workspace_bytes < need)
    return fail(TERRA_ERR_WORKSPACE, "workspace of %zu bytes given, %zu needed",
                workspace ? workspace_bytes : (size_t)0, need);
  return hip_status(terra::launch_attn_bwd(G, dtype, nhwc, q, k, v, o, o_lo, dout, lse,
                                           bias_table, dq, dk, dv, dbias_table, workspace,
                                           (hipStream_t)stream),
                    nhwc ? "terra_winattn_bwd_nhwc launch" : "terra_winattn_bwd launch");
}

extern "C" {

int terra_winattn_fwd(const terra_geom* g, int dtype, const void* q, const void* k, const void* v,
                      const float* bias_table, void* o, void* o_lo, float* lse, void* stream) {
  return attn_fwd_common(g, dtype, false, q, k, v, bias_table, o, o_lo, lse, stream);
}

int terra_winattn_fwd_nhwc(const terra_geom* g, int dtype, const void* q, const void* k,
                           const void* v, const float* bias_table, void* o, void* o_lo,
                           float* lse, void* stream) {
  return attn_fwd_common(g, dtype, true, q, k, v, bias_table, o, o_lo, lse, stream);
}

int terra_winattn_uses_o_lo(const terra_geom* g, int dtype) {
  int s = check_attn(g, dtype);
  if (s) return -s;
  ok();
  return terra::attn_uses_olo(make_geo(g), dtype) ? 1 : 0;
}

size_t terra_winattn_bwd_workspace_bytes(const terra_geom* g, int dtype) {
  if (check_attn(g, dtype)) return 0;
  return terra::bwd_workspace(make_geo(g), dtype);
}

int terra_winattn_bwd(const terra_geom* g, int dtype, const void* q, const void* k, const void* v,
                      const void* o, const void* o_lo, const void* dout, const float* lse,
                      const float* bias_table, void* dq, void* dk, void* dv, float* dbias_table,
                      void* workspace, size_t workspace_bytes, void* stream) {
  return attn_bwd_common(g, dtype, false, q, k, v, o, o_lo, dout, lse, bias_table, dq, dk, dv,
                         dbias_table, workspace, workspace_bytes, stream);
}

int terra_winattn_bwd_nhwc(const terra_geom* g, int dtype, const void* q, const void* k,
                           const void* v, const void* o, const void* o_lo, const void* dout,
                           const float* lse, const float* bias_table, void* dq, void* dk,
                           void* dv, float* dbias_table, void* workspace, size_t workspace_bytes,
                           void* stream) {
  return attn_bwd_common(g, dtype, true, q, k, v, o, o_lo, dout, lse, bias_table, dq, dk, dv,
                         dbias_table, workspace, workspace_bytes, stream);
}

}  // extern "C"

namespace {
int check_block(const terra_geom* g, int dtype) {
  int s = check_attn(g, dtype);
  if (s) return s;
  if (dtype != TERRA_BF16) return fail(TERRA_ERR_UNSUPPORTED, "the Swin block takes TERRA_BF16 only");
  if (g->C % 128 != 0 || g->C > 2048)
    return fail(TERRA_ERR_UNSUPPORTED, "the Swin block needs C a multiple of 128 and at most 2048 (C = %d)", g->C);
  if ((int64_t)g->B * g->H * g->W * 4 * g->C >= kMaxElems / 2)
    return fail(TERRA_ERR_UNSUPPORTED, "B*H*W*4C must be below 2^30 (operands under 2 GiB)");
  return ok();
}
terra::BlockParams to_params(const terra_block_params* p) {
  return terra::BlockParams{p->ln1_g, p->ln1_b, p->w_qkv, p->b_qkv, p->w_proj, p->b_proj,
                            p->ln2_g, p->ln2_b, p->w_fc1, p->b_fc1, p->w_fc2, p->b_fc2};
}
terra::BlockSaved to_saved(const terra_block_saved* v) {
  return terra::BlockSaved{v->mu1, v->rstd1, v->mu2, v->rstd2, v->q, v->k, v->v, v->o, v->lse, v->x1, v->h, v->a};
}
terra::BlockGrads to_grads(const terra_block_grads* g) {
  return terra::BlockGrads{g->ln1_g, g->ln1_b, g->w_qkv, g->b_qkv, g->w_proj, g->b_proj,
                           g->ln2_g, g->ln2_b, g->w_fc1, g->b_fc1, g->w_fc2, g->b_fc2};
}
bool any_null(std::initializer_list<const void*> ps) {
  for (const void* p : ps)
    if (!p) return true;
  return false;
}
}  // namespace

extern "C" {

size_t terra_block_fwd_workspace_bytes(const terra_geom* g, int dtype) {
  if (check_block(g, dtype)) return 0;
  return terra::block_fwd_workspace(make_geo(g));
}

int terra_block_fwd(const terra_geom* g, int dtype, const void* x, const terra_block_params* p,
                    const float* bias_table, void* x2, const terra_block_saved* sv, void* workspace,
                    size_t workspace_bytes, void* stream) {
  int s = check_block(g, dtype);
  if (s) return s;
  if (!p || !sv) return fail(TERRA_ERR_INVALID, "parameter or saved-activation struct is NULL");
  if (any_null({x, bias_table, x2, p->ln1_g, p->ln1_b, p->w_qkv, p->b_qkv, p->w_proj, p->b_proj, p->ln2_g,
                p->ln2_b, p->w_fc1, p->b_fc1, p->w_fc2, p->b_fc2, sv->mu1, sv->rstd1, sv->mu2, sv->rstd2, sv->q,
                sv->k, sv->v, sv->o, sv->lse, sv->x1, sv->h, sv->a}))
    return fail(TERRA_ERR_INVALID, "tensor pointer is NULL");
  const size_t need = terra::block_fwd_workspace(make_geo(g));
  if (!workspace || workspace_bytes < need)
    return fail(TERRA_ERR_WORKSPACE, "workspace of %zu bytes given, %zu needed", workspace ? workspace_bytes : (size_t)0,
                need);
  terra::Geo G = launch_geo(g);
  return hip_status(terra::launch_block_fwd(G, x, to_params(p), bias_table, x2, to_saved(sv), workspace,
                                            (hipStream_t)stream),
                    "terra_block_fwd launch");
}

size_t terra_block_bwd_workspace_bytes(const terra_geom* g, int dtype) {
  if (check_block(g, dtype)) return 0;
  return terra::block_bwd_workspace(make_geo(g));
}

int terra_block_bwd(const terra_geom* g, int dtype, const void* dx2, const void* x, const terra_block_params* p,
                    const float* bias_table, const terra_block_saved* sv, void* dx, const terra_block_grads* gr,
                    float* dbias_table, void* workspace, size_t workspace_bytes, void* stream) {
  int s = check_block(g, dtype);
  if (s) return s;
  if (!p || !sv || !gr) return fail(TERRA_ERR_INVALID, "parameter, saved-activation or gradient struct is NULL");
  if (any_null({dx2, x, bias_table, dx, dbias_table, p->ln1_g, p->ln1_b, p->w_qkv, p->b_qkv, p->w_proj, p->b_proj,
                p->ln2_g, p->ln2_b, p->w_fc1, p->b_fc1, p->w_fc2, p->b_fc2, sv->mu1, sv->rstd1, sv->mu2,
                sv->rstd2, sv->q, sv->k, sv->v, sv->o, sv->lse, sv->x1, sv->h, sv->a, gr->ln1_g, gr->ln1_b,
                gr->w_qkv, gr->b_qkv, gr->w_proj, gr->b_proj, gr->ln2_g, gr->ln2_b, gr->w_fc1, gr->b_fc1,
                gr->w_fc2, gr->b_fc2}))
    return fail(TERRA_ERR_INVALID, "tensor pointer is NULL");
  const size_t need = terra::block_bwd_workspace(make_geo(g));
  if (!workspace || workspace_bytes < need)
    return fail(TERRA_ERR_WORKSPACE, "workspace of %zu bytes given, %zu needed", workspace ? workspace_bytes : (size_t)0,
                need);
  terra::Geo G = launch_geo(g);
  return hip_status(terra::launch_block_bwd(G, dx2, x, to_params(p), bias_table, to_saved(sv), dx, to_grads(gr),
                                            dbias_table, workspace, (hipStream_t)stream),
                    "terra_block_bwd launch");
}

int terra_plan_padded_grid(int32_t H, int32_t W, int32_t p, int32_t alpha, int32_t w, int32_t m,
                           int32_t n, int32_t* Hhat, int32_t* What, double* overhead) {
  if (H < 1 || W < 1 || p < 1 || alpha < 1 || w < 1 || m < 1 || n < 1)
    return fail(TERRA_ERR_INVALID, "H, W, p, alpha, w, m and n must be >= 1");
  if (!Hhat || !What) return fail(TERRA_ERR_INVALID, "output pointer is NULL");
  int64_t hh, ww;
  terra::plan_padded(H, W, p, alpha, w, m, n, &hh, &ww);
  if (hh > INT32_MAX || ww > INT32_MAX) return fail(TERRA_ERR_UNSUPPORTED, "padded size exceeds 2^31-1");
  *Hhat = (int32_t)hh;
  *What = (int32_t)ww;
  if (overhead) *overhead = (double)hh * (double)ww / ((double)H * (double)W) - 1.0;
  return ok();
}

int terra_plan_window_ranges(int64_t M, int32_t ranks, int64_t* bounds) {
  if (M < 0 || ranks < 1) return fail(TERRA_ERR_INVALID, "need M >= 0 and ranks >= 1");
  if (!bounds) return fail(TERRA_ERR_INVALID, "output pointer is NULL");
  if (M > ((int64_t)1 << 40) || ranks > (1 << 20))
    return fail(TERRA_ERR_UNSUPPORTED, "M above 2^40 or more than 2^20 ranks");
  for (int32_t r = 0; r <= ranks; ++r) bounds[r] = terra::range_begin(M, ranks, r);
  return ok();
}

static int plan_common(const terra_geom* g, int32_t ranks, int32_t rank, terra::RankPlan* plan,
                       terra::Frag* frags) {
  int s = check_geom(g);
  if (s) return s;
  if (ranks < 1 || rank < 0 || rank >= ranks)
    return fail(TERRA_ERR_INVALID, "need ranks >= 1 and 0 <= rank (%d) < ranks (%d)", rank, ranks);
  if (ranks > 65536) return fail(TERRA_ERR_UNSUPPORTED, "more than 65536 ranks");
  terra::Geo G = make_geo(g);
  if (terra::plan_rank(G, ranks, rank, plan, frags, terra::kMaxFrags) < 0)
    return fail(TERRA_ERR_UNSUPPORTED,
                "rank %d of %d receives more than %d fragments (stripes much thinner than a window)",
                rank, ranks, terra::kMaxFrags);
  return ok();
}

int terra_plan_rank(const terra_geom* g, int32_t ranks, int32_t rank, terra_rank_plan* plan,
                    terra_fragment* frags) {
  if (!plan) return fail(TERRA_ERR_INVALID, "plan pointer is NULL");
  terra::RankPlan P;
  terra::Frag F[terra::kMaxFrags];
  int s = plan_common(g, ranks, rank, &P, F);
  if (s) return s;
  plan->win_begin = P.win_begin; plan->win_end = P.win_end;
  plan->slot_begin = P.slot_begin; plan->slot_end = P.slot_end;
  plan->row_begin = P.row_begin; plan->row_end = P.row_end;
  plan->nfrag = P.nfrag; plan->frag_tokens = P.frag_tokens;
  if (frags)
    for (int f = 0; f < P.nfrag; ++f) {
      frags[f].src_rank = F[f].src;
      frags[f].u0 = F[f].u0; frags[f].u1 = F[f].u1;
      frags[f].v0 = F[f].v0; frags[f].v1 = F[f].v1;
      frags[f].offset = F[f].offset;
    }
  return ok();
}

static int rank_route_common(const terra_geom* g, int dtype, int32_t ranks, int32_t rank,
                             void* stripe, void* frag_buf, void* y_win, bool forward, void* stream) {
  terra::RankPlan P;
  terra::Frag F[terra::kMaxFrags];
  int s = plan_common(g, ranks, rank, &P, F);
  if (s) return s;
  if ((s = check_dtype(dtype))) return s;
  const bool need_y = P.slot_end > P.slot_begin;
  if ((need_y && !y_win) || (P.row_end > P.row_begin && need_y && !stripe) ||
      (P.frag_tokens > 0 && !frag_buf))
    return fail(TERRA_ERR_INVALID, "tensor pointer is NULL");
  const int esize = dtype == TERRA_F32 ? 4 : 2;
  const int64_t row_bytes = (int64_t)g->C * esize;
  if ((int64_t)g->wh * g->ww * (row_bytes / 2) >= ((int64_t)1 << 22))
    return fail(TERRA_ERR_UNSUPPORTED, "window of %d tokens x %lld bytes is too large to route",
                g->wh * g->ww, (long long)row_bytes);
  terra::Geo G = make_geo(g);
  return hip_status(terra::launch_route_rank(G, (int)row_bytes, P, F, stripe, frag_buf, y_win, forward,
                                             (hipStream_t)stream),
                    forward ? "terra_window_route_rank launch" : "terra_window_unroute_rank launch");
}

int terra_window_route_rank(const terra_geom* g, int dtype, int32_t ranks, int32_t rank,
                            const void* stripe, const void* frag_buf, void* y_win, void* stream) {
  return rank_route_common(g, dtype, ranks, rank, const_cast<void*>(stripe),
                           const_cast<void*>(frag_buf), y_win, true, stream);
}

int terra_window_unroute_rank(const terra_geom* g, int dtype, int32_t ranks, int32_t rank,
                              const void* y_win, void* stripe, void* frag_buf, void* stream) {
  return rank_route_common(g, dtype, ranks, rank, stripe, frag_buf, const_cast<void*>(y_win), false,
                           stream);
}

static int frag_common(const terra_geom* g, int dtype, int32_t ranks, int32_t dst_rank,
                       int32_t src_rank, void* src_stripe, void* frag_buf, bool pack, void* stream) {
  terra::RankPlan P;
  terra::Frag F[terra::kMaxFrags];
  int s = plan_common(g, ranks, dst_rank, &P, F);
  if (s) return s;
  if ((s = check_dtype(dtype))) return s;
  if (src_rank < 0 || src_rank >= ranks)
    return fail(TERRA_ERR_INVALID, "src_rank %d outside [0, %d)", src_rank, ranks);
  bool any = false;
  for (int f = 0; f < P.nfrag; ++f) any = any || F[f].src == src_rank;
  if (!any) return ok();
  if (!src_stripe || !frag_buf) return fail(TERRA_ERR_INVALID, "tensor pointer is NULL");
  if (src_stripe == frag_buf) return fail(TERRA_ERR_INVALID, "stripe and fragment buffer must differ");
  const int esize = dtype == TERRA_F32 ? 4 : 2;
  terra::Geo G = make_geo(g);
  return hip_status(terra::launch_frag_copy(G, g->C * esize, P, F, src_rank,
                                            terra::stripe_begin(g->H, ranks, src_rank),
                                            terra::stripe_begin(g->H, ranks, src_rank + 1), src_stripe,
                                            frag_buf, pack, (hipStream_t)stream),
                    pack ? "terra_fragment_pack launch" : "terra_fragment_unpack launch");
}

int terra_fragment_pack(const terra_geom* g, int dtype, int32_t ranks, int32_t dst_rank,
                        int32_t src_rank, const void* src_stripe, void* frag_buf, void* stream) {
  return frag_common(g, dtype, ranks, dst_rank, src_rank, const_cast<void*>(src_stripe), frag_buf,
                     true, stream);
}

int terra_fragment_unpack(const terra_geom* g, int dtype, int32_t ranks, int32_t dst_rank,
                          int32_t src_rank, const void* frag_buf, void* src_stripe, void* stream) {
  return frag_common(g, dtype, ranks, dst_rank, src_rank, src_stripe, const_cast<void*>(frag_buf),
                     false, stream);
}

}  // extern "C"

// Device memory of the allocation-free backward: one array per GPU, held
// until the process ends.  Its name is a host-side stand-in in host code;
// the device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[TERRA_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Address of the current device's scratch array (set up on first use).
int scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(TERRA_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(TERRA_ERR_UNSUPPORTED, "device %d >= %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(TERRA_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return ok();
}
}  // namespace

extern "C" {

int terra_winattn_bwd_nhwc_noalloc(const terra_geom* g, int dtype, const void* q, const void* k,
                                   const void* v, const void* o, const void* o_lo,
                                   const void* dout, const float* lse, const float* bias_table,
                                   void* dq, void* dk, void* dv, float* dbias_table,
                                   void* stream) {
  int s = check_attn(g, dtype);
  if (s) return s;
  const size_t need = terra::bwd_workspace(make_geo(g), dtype);
  if (need > (size_t)TERRA_SCRATCH_BYTES)
    return fail(TERRA_ERR_UNSUPPORTED,
                "this geometry needs %zu bytes of scratch; the library holds %zu per GPU "
                "(use terra_winattn_bwd_nhwc with a workspace)",
                need, (size_t)TERRA_SCRATCH_BYTES);
  void* ws = nullptr;
  if ((s = scratch_address(&ws))) return s;
  return attn_bwd_common(g, dtype, true, q, k, v, o, o_lo, dout, lse, bias_table, dq, dk, dv,
                         dbias_table, ws, (size_t)TERRA_SCRATCH_BYTES, stream);
}

const char* terra_status_string(int status) {
  switch (status) {
    case TERRA_OK: return "ok";
    case TERRA_ERR_INVALID: return "invalid argument";
    case TERRA_ERR_UNSUPPORTED: return "unsupported";
    case TERRA_ERR_WORKSPACE: return "workspace too small";
    case TERRA_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* terra_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
