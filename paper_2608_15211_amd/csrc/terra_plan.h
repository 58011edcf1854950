// terra_plan.h - ragged window assignment and per-rank route plan shared by
// the host planner (plan.hip), the rank-local route kernels (route.hip) and
// the C ABI (abi.hip).
#pragma once

#include <stdint.h>

namespace terra {

struct Geo;

// Most fragments one rank may receive: the rank's windows cover at most
// three rectangles of the rolled grid, each at most four of the original
// grid, cut by the stripes they cross; 64 covers every split in which a
// window row is at most a few stripes tall.
constexpr int kMaxFrags = 64;

// One rectangle of the token grid that a rank receives from another:
// rows [u0, u1), columns [v0, v1) of the original grid, held by DMP rank
// src, stored row-major from token `offset` of the receiver's fragment
// buffer (per image).
struct Frag {
  int src, u0, u1, v0, v1, offset;
};

struct RankPlan {
  int win_begin, win_end;     // Eq. (4) window range [L_r, R_r)
  int slot_begin, slot_end;   // its window-major token slots (one image)
  int row_begin, row_end;     // DMP stripe rows held by the rank
  int nfrag;                  // fragments received from other ranks
  int frag_tokens;            // tokens per image in the fragment buffer
};

void plan_padded(int64_t H, int64_t W, int64_t p, int64_t alpha, int64_t w, int64_t m, int64_t n,
                 int64_t* Hhat, int64_t* What);
int64_t range_begin(int64_t M, int64_t ranks, int64_t r);
int stripe_begin(int H, int ranks, int r);
int plan_rank(const Geo& g, int ranks, int rank, RankPlan* plan, Frag* frags, int cap);

}  // namespace terra
