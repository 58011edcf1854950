// plan.hip - host-side planner of the ragged window assignment (Sec. V-A)
// and of the per-rank token route with its boundary fragments (Sec. IV-D).
//
// Pure host code: closed forms of Eq. (3) and Eq. (4), the DMP height
// stripes of the I/O topology (Sec. IV-B), and, for one rank, the list of
// rectangles of the token grid that its route needs from other ranks.
#include <algorithm>
#include <vector>

#include "terra_common.h"
#include "terra_plan.h"

namespace terra {

// Eq. (3): the least multiple of p*alpha*w*m (p*alpha*w*n) not below H (W).
void plan_padded(int64_t H, int64_t W, int64_t p, int64_t alpha, int64_t w, int64_t m, int64_t n,
                 int64_t* Hhat, int64_t* What) {
  const int64_t uh = p * alpha * w * m, uw = p * alpha * w * n;
  *Hhat = (H + uh - 1) / uh * uh;
  *What = (W + uw - 1) / uw * uw;
}

// Eq. (4): first window of rank r under the ragged Topo(ranks, 1); rank r
// owns [range_begin(r), range_begin(r + 1)).
int64_t range_begin(int64_t M, int64_t ranks, int64_t r) { return r * M / ranks; }

// DMP stripes: rank r holds grid rows [stripe_begin(r), stripe_begin(r + 1)),
// the floor rule of Eq. (4) applied to rows (equal stripes when ranks
// divides H, as on the paper's padded grids).
int stripe_begin(int H, int ranks, int r) { return (int)((int64_t)r * H / ranks); }

namespace {

struct Rect { int src, u0, u1, v0, v1; };

// [x0, x1) shifted by s on a cycle of length n (x1 <= n): one or two intervals.
int cyc_split(int x0, int x1, int s, int n, int out[2][2]) {
  const int a = x0 + s, b = x1 + s;
  if (b <= n) { out[0][0] = a; out[0][1] = b; return 1; }
  if (a >= n) { out[0][0] = a - n; out[0][1] = b - n; return 1; }
  out[0][0] = a; out[0][1] = n;
  out[1][0] = 0; out[1][1] = b - n;
  return 2;
}

bool try_merge(Rect& a, const Rect& b) {
  if (a.src != b.src) return false;
  if (a.u0 == b.u0 && a.u1 == b.u1) {
    if (a.v1 == b.v0) { a.v1 = b.v1; return true; }
    if (b.v1 == a.v0) { a.v0 = b.v0; return true; }
  }
  if (a.v0 == b.v0 && a.v1 == b.v1) {
    if (a.u1 == b.u0) { a.u1 = b.u1; return true; }
    if (b.u1 == a.u0) { a.u0 = b.u0; return true; }
  }
  return false;
}

}  // namespace

// Plan of rank `rank` among `ranks`.  The rank's windows (row-major range of
// Eq. (4)) cover, in the rolled grid, at most three rectangles: the tail of
// its first window row, whole window rows, and the head of its last window
// row.  Undoing the shift maps each to at most four rectangles of the
// original grid (the rows and the columns may each wrap once); those are cut
// by the DMP stripes, and the pieces held by other ranks are the fragments
// the rank receives.  Fragments are merged where they share a source and an
// edge, and sorted by source rank, so that everything one source sends to
// the rank is one contiguous run of the fragment buffer.
// Returns the fragment count, or -1 if more than `cap`.
int plan_rank(const Geo& g, int ranks, int rank, RankPlan* plan, Frag* frags, int cap) {
  const int64_t M = (int64_t)g.Mh * g.Mw;
  const int64_t L = range_begin(M, ranks, rank), R = range_begin(M, ranks, rank + 1);
  plan->win_begin = (int)L;
  plan->win_end = (int)R;
  auto slot_of = [&](int64_t w) -> int {
    if (w >= M) return g.HW;
    const int i = (int)(w / g.Mw), j = (int)(w - (int64_t)i * g.Mw);
    return win_offset(g, i, j);
  };
  plan->slot_begin = slot_of(L);
  plan->slot_end = slot_of(R);
  plan->row_begin = stripe_begin(g.H, ranks, rank);
  plan->row_end = stripe_begin(g.H, ranks, rank + 1);
  plan->nfrag = 0;
  plan->frag_tokens = 0;
  if (L == R) return 0;

  // rolled-grid rectangles in window units: (i0, i1, j0, j1)
  int pieces[3][4];
  int np = 0;
  const int ia = (int)(L / g.Mw), ja = (int)(L % g.Mw);
  const int ib = (int)((R - 1) / g.Mw), jb = (int)((R - 1) % g.Mw);
  auto add = [&](int i0, int i1, int j0, int j1) {
    pieces[np][0] = i0; pieces[np][1] = i1; pieces[np][2] = j0; pieces[np][3] = j1;
    ++np;
  };
  if (ia == ib) {
    add(ia, ia + 1, ja, jb + 1);
  } else {
    add(ia, ia + 1, ja, g.Mw);
    if (ib > ia + 1) add(ia + 1, ib, 0, g.Mw);
    add(ib, ib + 1, 0, jb + 1);
  }

  std::vector<Rect> rects;
  for (int p = 0; p < np; ++p) {
    const int r0 = pieces[p][0] * g.wh, r1 = std::min(pieces[p][1] * g.wh, g.H);
    const int c0 = pieces[p][2] * g.ww, c1 = std::min(pieces[p][3] * g.ww, g.W);
    int rows[2][2], cols[2][2];
    const int nr = cyc_split(r0, r1, g.sh, g.H, rows);
    const int nc = cyc_split(c0, c1, g.sw, g.W, cols);
    for (int a = 0; a < nr; ++a)
      for (int s = 0; s < ranks; ++s) {
        const int u0 = std::max(rows[a][0], stripe_begin(g.H, ranks, s));
        const int u1 = std::min(rows[a][1], stripe_begin(g.H, ranks, s + 1));
        if (u0 >= u1 || s == rank) continue;
        for (int c = 0; c < nc; ++c) rects.push_back(Rect{s, u0, u1, cols[c][0], cols[c][1]});
      }
  }
  for (bool merged = true; merged;) {
    merged = false;
    for (size_t x = 0; x < rects.size() && !merged; ++x)
      for (size_t y = x + 1; y < rects.size() && !merged; ++y)
        if (try_merge(rects[x], rects[y])) {
          rects.erase(rects.begin() + y);
          merged = true;
        }
  }
  std::sort(rects.begin(), rects.end(), [](const Rect& a, const Rect& b) {
    if (a.src != b.src) return a.src < b.src;
    if (a.u0 != b.u0) return a.u0 < b.u0;
    return a.v0 < b.v0;
  });
  if ((int)rects.size() > cap) return -1;
  int64_t off = 0;
  for (size_t x = 0; x < rects.size(); ++x) {
    frags[x].src = rects[x].src;
    frags[x].u0 = rects[x].u0;
    frags[x].u1 = rects[x].u1;
    frags[x].v0 = rects[x].v0;
    frags[x].v1 = rects[x].v1;
    frags[x].offset = (int)off;
    off += (int64_t)(rects[x].u1 - rects[x].u0) * (rects[x].v1 - rects[x].v0);
  }
  plan->nfrag = (int)rects.size();
  plan->frag_tokens = (int)off;
  return plan->nfrag;
}

}  // namespace terra
