// route.hip - token route between the NHWC layout and the window-major
// layout, and its inverse (Sec. IV-D: the route gathers each token into its
// window-major slot after the window shift; the inverse route scatters it
// back and is the route's backward).
//
// Pure HBM streaming: every token row (C elements) moves once in each
// direction.  A workgroup copies a contiguous part of one window; inside a
// window, the tokens of one window row come from a contiguous run of the
// source row (two runs where the run crosses the longitude edge), so loads
// and stores are wide (16 B per lane) and coalesced.
#include "terra_common.h"
#include "terra_plan.h"

#include <algorithm>
#include <initializer_list>

namespace terra {

template <int VEC> struct VecT;
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
template <> struct VecT<16> { typedef u32x4_t type; };
template <> struct VecT<8> { typedef u32x2_t type; };
template <> struct VecT<4> { typedef uint32_t type; };
template <> struct VecT<2> { typedef uint16_t type; };

struct RouteArgs {
  Geo g;
  int cpr;          // VEC-sized chunks per token row
  float rcp_cpr;
  int split;        // workgroups per window
};

constexpr int kRouteThreads = 256;
constexpr int kRouteUnroll = 1;

// FORWARD=true: NHWC -> window-major.  FORWARD=false: window-major -> NHWC.
template <int VEC, bool FORWARD>
__global__ __launch_bounds__(kRouteThreads) void route_kernel(
    const typename VecT<VEC>::type* __restrict__ src,
    typename VecT<VEC>::type* __restrict__ dst, RouteArgs A) {
  typedef typename VecT<VEC>::type V;
  const Geo& g = A.g;
  const int wid = blockIdx.x / A.split;
  const int part = blockIdx.x - wid * A.split;
  const int b = wid / g.nwin;
  const int w = wid - b * g.nwin;
  const int i = w / g.Mw;
  const int j = w - i * g.Mw;
  const int rows = win_rows(g, i);
  const int cols = win_cols(g, j);
  const int off = win_offset(g, i, j);
  const float rcp_cols = 1.0f / (float)cols;
  const int nchunk = rows * cols * A.cpr;
  const int step = kRouteThreads * kRouteUnroll;
  const int per = ((nchunk + A.split - 1) / A.split + step - 1) / step * step;
  const int start = part * per;
  const int end = min(nchunk, start + per);
  const int64_t img_base = (int64_t)b * g.HW;

  for (int k0 = start + threadIdx.x; k0 < end; k0 += step) {
    V val[kRouteUnroll];
    int64_t nhwc[kRouteUnroll], win[kRouteUnroll];
#pragma unroll
    for (int u = 0; u < kRouteUnroll; ++u) {
      const int k = k0 + u * kRouteThreads;
      const int t = fast_div(k, A.cpr, A.rcp_cpr);      // token within window
      const int ch = k - t * A.cpr;
      const int a = fast_div(t, cols, rcp_cols);          // in-window row
      const int c = t - a * cols;                         // in-window column
      int r = i * g.wh + a + g.sh;                        // original row
      if (r >= g.H) r -= g.H;
      int s = j * g.ww + c + g.sw;                        // original column
      if (s >= g.W) s -= g.W;
      nhwc[u] = ((img_base + (int64_t)r * g.W + s) * A.cpr) + ch;
      win[u] = ((img_base + off + t) * (int64_t)A.cpr) + ch;
      if (k < end) {
        val[u] = FORWARD ? __builtin_nontemporal_load(src + nhwc[u])
                         : __builtin_nontemporal_load(src + win[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < kRouteUnroll; ++u) {
      const int k = k0 + u * kRouteThreads;
      if (k < end) {
        if (FORWARD) __builtin_nontemporal_store(val[u], dst + win[u]);
        else __builtin_nontemporal_store(val[u], dst + nhwc[u]);
      }
    }
  }
}

// Window-major layout of one image on the device: offsets[w] (w <= nwin,
// offsets[nwin] = H*W) and counts[w] (w < nwin); either may be null.
__global__ __launch_bounds__(kRouteThreads) void layout_kernel(Geo g, int32_t* offsets,
                                                               int32_t* counts) {
  const int w = blockIdx.x * kRouteThreads + threadIdx.x;
  if (w > g.nwin) return;
  if (w == g.nwin) {
    if (offsets) offsets[w] = g.HW;
    return;
  }
  const int i = w / g.Mw, j = w - (w / g.Mw) * g.Mw;
  if (offsets) offsets[w] = win_offset(g, i, j);
  if (counts) counts[w] = win_rows(g, i) * win_cols(g, j);
}

hipError_t launch_layout(const Geo& g, int32_t* offsets, int32_t* counts, hipStream_t stream) {
  const int grid = (g.nwin + 1 + kRouteThreads - 1) / kRouteThreads;
  hipLaunchKernelGGL(layout_kernel, dim3(grid), dim3(kRouteThreads), 0, stream, g, offsets, counts);
  return hipGetLastError();
}

template <int VEC>
static hipError_t launch_route_vec(const RouteArgs& A, const void* src, void* dst,
                                   bool forward, hipStream_t stream) {
  typedef typename VecT<VEC>::type V;
  const int grid = A.g.B * A.g.nwin * A.split;
  if (forward)
    hipLaunchKernelGGL((route_kernel<VEC, true>), dim3(grid), dim3(kRouteThreads), 0, stream,
                       (const V*)src, (V*)dst, A);
  else
    hipLaunchKernelGGL((route_kernel<VEC, false>), dim3(grid), dim3(kRouteThreads), 0, stream,
                       (const V*)src, (V*)dst, A);
  return hipGetLastError();
}

// Host entry used by the C ABI.  row_bytes = C * element size.
hipError_t launch_route(const Geo& g, int row_bytes, const void* src, void* dst,
                        bool forward, hipStream_t stream) {
  RouteArgs A;
  A.g = g;
  int vec = 2;
  if (row_bytes % 16 == 0 && ((uintptr_t)src % 16 == 0) && ((uintptr_t)dst % 16 == 0)) vec = 16;
  else if (row_bytes % 8 == 0 && ((uintptr_t)src % 8 == 0) && ((uintptr_t)dst % 8 == 0)) vec = 8;
  else if (row_bytes % 4 == 0 && ((uintptr_t)src % 4 == 0) && ((uintptr_t)dst % 4 == 0)) vec = 4;
  A.cpr = row_bytes / vec;
  A.rcp_cpr = 1.0f / (float)A.cpr;
  // Many short workgroups (one 16-byte chunk per thread, up to ~64K
  // workgroups) keep more loads in flight across the chip than fewer long
  // ones: 6.4 TB/s against 5.6 TB/s with 4K workgroups of four chunks per
  // thread on a 212 MB tensor.
  const int64_t chunks_per_win = (int64_t)g.wh * g.ww * A.cpr;
  const int64_t nwin_total = (int64_t)g.B * g.nwin;
  int split = (int)((65536 + nwin_total - 1) / nwin_total);
  const int64_t max_split = (chunks_per_win + kRouteThreads * kRouteUnroll - 1) /
                            (kRouteThreads * kRouteUnroll);
  if (split > max_split) split = (int)max_split;
  if (split < 1) split = 1;
  A.split = split;
  switch (vec) {
    case 16: return launch_route_vec<16>(A, src, dst, forward, stream);
    case 8: return launch_route_vec<8>(A, src, dst, forward, stream);
    case 4: return launch_route_vec<4>(A, src, dst, forward, stream);
    default: return launch_route_vec<2>(A, src, dst, forward, stream);
  }
}


// ---------------------------------------------------------------------------
// Per-rank route (Sec. IV-D with the ragged window ranges of Sec. V-A,
// Eq. (4)).  Rank r owns windows [L_r, R_r) of every image and the DMP
// stripe of grid rows [row_begin, row_end).  Its route fills the
// window-major slots of its windows from its own stripe and from the
// fragment buffer, which holds the rectangles of the grid that other ranks
// send it (the shift route's boundary fragments); its inverse scatters them
// back to the same places (the route's backward).
// ---------------------------------------------------------------------------
struct RankRouteArgs {
  Geo g;
  int cpr;          // VEC-sized chunks per token row
  float rcp_cpr;
  int split;        // workgroups per window
  int win_begin, nwin;    // the rank's windows
  int slot_begin, ntok;   // their slots [slot_begin, slot_begin + ntok) per image
  int row_begin, nrows;   // the rank's stripe
  int ftok, nfrag;        // fragment buffer tokens per image, fragment count
  Frag frag[kMaxFrags];
};

// FORWARD=true: stripe + fragments -> window-major; false: the inverse.
template <int VEC, bool FORWARD>
__global__ __launch_bounds__(kRouteThreads) void route_rank_kernel(
    typename VecT<VEC>::type* __restrict__ stripe, typename VecT<VEC>::type* __restrict__ fbuf,
    typename VecT<VEC>::type* __restrict__ y, RankRouteArgs A) {
  typedef typename VecT<VEC>::type V;
  const Geo& g = A.g;
  const int wid = blockIdx.x / A.split;
  const int part = blockIdx.x - wid * A.split;
  const int b = wid / A.nwin;
  const int w = A.win_begin + (wid - b * A.nwin);
  const int i = w / g.Mw;
  const int j = w - i * g.Mw;
  const int rows = win_rows(g, i);
  const int cols = win_cols(g, j);
  const int off = win_offset(g, i, j) - A.slot_begin;
  const float rcp_cols = 1.0f / (float)cols;
  const int nchunk = rows * cols * A.cpr;
  const int per = ((nchunk + A.split - 1) / A.split + kRouteThreads - 1) / kRouteThreads * kRouteThreads;
  const int start = part * per;
  const int end = min(nchunk, start + per);

  for (int k = start + threadIdx.x; k < end; k += kRouteThreads) {
    const int t = fast_div(k, A.cpr, A.rcp_cpr);
    const int ch = k - t * A.cpr;
    const int a = fast_div(t, cols, rcp_cols);
    const int c = t - a * cols;
    int u = i * g.wh + a + g.sh;
    if (u >= g.H) u -= g.H;
    int v = j * g.ww + c + g.sw;
    if (v >= g.W) v -= g.W;
    const int64_t yi = ((int64_t)b * A.ntok + off + t) * A.cpr + ch;
    V* base = nullptr;
    int64_t si = 0;
    if ((unsigned)(u - A.row_begin) < (unsigned)A.nrows) {
      base = stripe;
      si = (((int64_t)b * A.nrows + (u - A.row_begin)) * g.W + v) * A.cpr + ch;
    } else {
      for (int f = 0; f < A.nfrag; ++f) {
        const Frag& F = A.frag[f];
        if (u >= F.u0 && u < F.u1 && v >= F.v0 && v < F.v1) {
          base = fbuf;
          si = ((int64_t)b * A.ftok + F.offset + (int64_t)(u - F.u0) * (F.v1 - F.v0) + (v - F.v0)) *
                   A.cpr + ch;
          break;
        }
      }
    }
    if (base == nullptr) continue;   // not reachable for a consistent plan
    if (FORWARD) __builtin_nontemporal_store(__builtin_nontemporal_load(base + si), y + yi);
    else __builtin_nontemporal_store(__builtin_nontemporal_load(y + yi), base + si);
  }
}

// The sender's side of the exchange: copy the fragments rank `dst` receives
// from rank `src` out of src's stripe into dst's fragment buffer (PACK), or
// back (the backward).  Fragments of one source are consecutive in the
// plan, so they form one contiguous run of the buffer: one message per pair
// of ranks on a multi-GPU system.
struct FragCopyArgs {
  int W, cpr, split;
  int frag_begin, nfrag;  // the run of fragments from src
  int row_begin, nrows;   // src's stripe
  int ftok;               // fragment buffer tokens per image
  Frag frag[kMaxFrags];
};

template <int VEC, bool PACK>
__global__ __launch_bounds__(kRouteThreads) void frag_copy_kernel(
    typename VecT<VEC>::type* __restrict__ stripe, typename VecT<VEC>::type* __restrict__ fbuf,
    FragCopyArgs A) {
  const int wid = blockIdx.x / A.split;
  const int part = blockIdx.x - wid * A.split;
  const int b = wid / A.nfrag;
  const Frag& F = A.frag[A.frag_begin + (wid - b * A.nfrag)];
  const int fw = F.v1 - F.v0;
  const int nchunk = (F.u1 - F.u0) * fw * A.cpr;
  const int per = ((nchunk + A.split - 1) / A.split + kRouteThreads - 1) / kRouteThreads * kRouteThreads;
  const int start = part * per;
  const int end = min(nchunk, start + per);
  for (int k = start + threadIdx.x; k < end; k += kRouteThreads) {
    const int t = k / A.cpr;
    const int ch = k - t * A.cpr;
    const int ru = t / fw;
    const int rv = t - ru * fw;
    const int64_t si = (((int64_t)b * A.nrows + (F.u0 + ru - A.row_begin)) * A.W + F.v0 + rv) * A.cpr + ch;
    const int64_t fi = ((int64_t)b * A.ftok + F.offset + t) * A.cpr + ch;
    if (PACK) __builtin_nontemporal_store(__builtin_nontemporal_load(stripe + si), fbuf + fi);
    else __builtin_nontemporal_store(__builtin_nontemporal_load(fbuf + fi), stripe + si);
  }
}

static int route_vec(int row_bytes, std::initializer_list<const void*> ptrs) {
  for (int vec : {16, 8, 4}) {
    bool ok = row_bytes % vec == 0;
    for (const void* p : ptrs) ok = ok && ((uintptr_t)p % vec == 0);
    if (ok) return vec;
  }
  return 2;
}

template <int VEC>
static void launch_rank_vec(RankRouteArgs& A, int grid, void* stripe, void* fbuf, void* y,
                            bool forward, hipStream_t st) {
  typedef typename VecT<VEC>::type V;
  if (forward)
    hipLaunchKernelGGL((route_rank_kernel<VEC, true>), dim3(grid), dim3(kRouteThreads), 0, st,
                       (V*)stripe, (V*)fbuf, (V*)y, A);
  else
    hipLaunchKernelGGL((route_rank_kernel<VEC, false>), dim3(grid), dim3(kRouteThreads), 0, st,
                       (V*)stripe, (V*)fbuf, (V*)y, A);
}

hipError_t launch_route_rank(const Geo& g, int row_bytes, const RankPlan& plan, const Frag* frags,
                             void* stripe, void* fbuf, void* y, bool forward, hipStream_t st) {
  const int nwin = plan.win_end - plan.win_begin;
  if (nwin == 0) return hipSuccess;
  RankRouteArgs A;
  A.g = g;
  const int vec = route_vec(row_bytes, {stripe, fbuf, y});
  A.cpr = row_bytes / vec;
  A.rcp_cpr = 1.0f / (float)A.cpr;
  const int64_t chunks_per_win = (int64_t)g.wh * g.ww * A.cpr;
  const int64_t nw = (int64_t)g.B * nwin;
  int64_t split = (65536 + nw - 1) / nw;
  const int64_t max_split = (chunks_per_win + kRouteThreads - 1) / kRouteThreads;
  A.split = (int)std::max<int64_t>(1, std::min(split, max_split));
  A.win_begin = plan.win_begin;
  A.nwin = nwin;
  A.slot_begin = plan.slot_begin;
  A.ntok = plan.slot_end - plan.slot_begin;
  A.row_begin = plan.row_begin;
  A.nrows = plan.row_end - plan.row_begin;
  A.ftok = plan.frag_tokens;
  A.nfrag = plan.nfrag;
  for (int f = 0; f < plan.nfrag; ++f) A.frag[f] = frags[f];
  const int grid = (int)(nw * A.split);
  switch (vec) {
    case 16: launch_rank_vec<16>(A, grid, stripe, fbuf, y, forward, st); break;
    case 8: launch_rank_vec<8>(A, grid, stripe, fbuf, y, forward, st); break;
    case 4: launch_rank_vec<4>(A, grid, stripe, fbuf, y, forward, st); break;
    default: launch_rank_vec<2>(A, grid, stripe, fbuf, y, forward, st); break;
  }
  return hipGetLastError();
}

template <int VEC>
static void launch_frag_vec(FragCopyArgs& A, int grid, void* stripe, void* fbuf, bool pack,
                            hipStream_t st) {
  typedef typename VecT<VEC>::type V;
  if (pack)
    hipLaunchKernelGGL((frag_copy_kernel<VEC, true>), dim3(grid), dim3(kRouteThreads), 0, st,
                       (V*)stripe, (V*)fbuf, A);
  else
    hipLaunchKernelGGL((frag_copy_kernel<VEC, false>), dim3(grid), dim3(kRouteThreads), 0, st,
                       (V*)stripe, (V*)fbuf, A);
}

// Copy between src's stripe and dst's fragment buffer every fragment of
// dst's plan whose source is src.  src_rows: [row_begin, row_end) of src.
hipError_t launch_frag_copy(const Geo& g, int row_bytes, const RankPlan& plan, const Frag* frags,
                            int src, int src_row_begin, int src_row_end, void* stripe, void* fbuf,
                            bool pack, hipStream_t st) {
  int fa = 0;
  while (fa < plan.nfrag && frags[fa].src != src) ++fa;
  int fb = fa;
  int64_t most = 0;
  while (fb < plan.nfrag && frags[fb].src == src) {
    most = std::max<int64_t>(most, (int64_t)(frags[fb].u1 - frags[fb].u0) * (frags[fb].v1 - frags[fb].v0));
    ++fb;
  }
  if (fb == fa) return hipSuccess;
  FragCopyArgs A;
  const int vec = route_vec(row_bytes, {stripe, fbuf});
  A.W = g.W;
  A.cpr = row_bytes / vec;
  A.frag_begin = fa;
  A.nfrag = fb - fa;
  A.row_begin = src_row_begin;
  A.nrows = src_row_end - src_row_begin;
  A.ftok = plan.frag_tokens;
  for (int f = 0; f < plan.nfrag; ++f) A.frag[f] = frags[f];
  const int64_t chunks = most * A.cpr;
  const int64_t nitems = (int64_t)g.B * A.nfrag;
  int64_t split = (chunks + 4 * kRouteThreads - 1) / (4 * kRouteThreads);
  A.split = (int)std::max<int64_t>(1, split);
  const int grid = (int)(nitems * A.split);
  switch (vec) {
    case 16: launch_frag_vec<16>(A, grid, stripe, fbuf, pack, st); break;
    case 8: launch_frag_vec<8>(A, grid, stripe, fbuf, pack, st); break;
    case 4: launch_frag_vec<4>(A, grid, stripe, fbuf, pack, st); break;
    default: launch_frag_vec<2>(A, grid, stripe, fbuf, pack, st); break;
  }
  return hipGetLastError();
}

}  // namespace terra
