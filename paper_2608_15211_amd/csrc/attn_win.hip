// attn_win.hip - window-resident attention kernels for windows of at most
// 128 tokens (bf16), the common Swin case (e.g. 8x8, 8x16 windows).
//
// Same mathematics as attn.hip (W-MSA / SW-MSA of the Swin blocks,
// Sec. IV-A, on the window-major layout of Sec. IV-D), organised so that a
// workgroup holds one whole window of one head:
// * every key of the window is in LDS at once: D_q = sum_k P dP is a
//   register sum over the window in the backward;
// * row-major tiles in LDS give their transposed operands through the LDS
//   transpose read (V for PV, K for dQ, Q and dO for dK and dV), and blocks
//   held in registers (P^T, dS^T for dV/dK) are transposed ON THE MATRIX
//   CORES: multiplying a block by a 0/1 permutation operand returns it in
//   the transposed register layout (values are exact bf16, so the copy is
//   exact);
// * the backward walks many windows of one head per workgroup, sums the
//   per-key partial dK/dV of its four waves in LDS in a fixed rotation, and
//   keeps per-wave bias-gradient bins in LDS, so that every result is
//   produced in a fixed order (bit-reproducible).
#include "terra_common.h"

namespace terra {

typedef __bf16 bf16;
constexpr int kWinThreads = 256;
constexpr int kWinMax = 128;      // tokens per window handled here
constexpr int kLabBadW = 0xFF;

__device__ inline int pi_slot(int s, int h) { return 8 * (s / 4) + 4 * h + (s % 4); }

// 0/1 operand that maps contraction chunk c onto output columns.
// PERM = true: the source block comes from result registers (slot s of half
// h is row 16c + pi_slot(s, h)); PERM = false: the source is a row of
// memory (slot s of half h is element 16c + 8h + s).
template <bool PERM>
__device__ inline bf16x8 ident_op(int c) {
  const int lane = threadIdx.x & 63;
  const int h = lane >> 5, col = lane & 31;
  bf16x8 o;
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    const int src = 16 * c + (PERM ? pi_slot(s, h) : 8 * h + s);
    o[s] = (bf16)(src == col ? 1.0f : 0.0f);
  }
  return o;
}

// Transpose of a 32x32 block given as two operands (chunks c = 0, 1).
__device__ inline f32x16 mfma_transpose(const bf16x8& a0, const bf16x8& a1, const bf16x8& i0,
                                        const bf16x8& i1) {
  f32x16 d = f32x16{};
  mma16(d, a0, i0);
  mma16(d, a1, i1);
  return d;
}

__device__ inline int win_token_info(const Geo& g, int i, int j, int cols, int t, int n) {
  if (t >= n) return kLabBadW << 24;
  const int a = fast_div(t, cols, win_rcols(g, j));
  const int c = t - a * cols;
  const int lab = row_label(g, i * g.wh + a) | col_label(g, j * g.ww + c);
  return (a * g.tstride + c) | (lab << 24);
}

// Entry x of the LDS bias table of head h: bins in reversed order, rows of
// tstride entries (the padding entries are never read), times `scale`; four
// -inf entries at ntab .. ntab+3 serve excluded pairs.
__device__ inline float table_entry(const Geo& g, const float* __restrict__ table, int h, int x,
                                    float scale) {
  if (x >= g.ntab) return -INFINITY;
  const int y = g.ntab - 1 - x;
  const int da = y / g.tstride, dc = y - da * g.tstride;
  return dc < g.bstride ? table[(da * g.bstride + dc) * g.heads + h] * scale : 0.0f;
}

// Reversed table index of query word qinf against key offset 0.
__device__ inline int table_qrev(const Geo& g, int qinf) {
  return g.ntab - 1 - ((qinf & 0xFFFFFF) + (g.wh - 1) * g.tstride + (g.ww - 1));
}

__device__ inline bf16x8 zero8() {
  bf16x8 z;
#pragma unroll
  for (int s = 0; s < 8; ++s) z[s] = (bf16)0.0f;
  return z;
}

// Store 4 consecutive floats of result registers 4g..4g+3 as bf16 (8 bytes).
__device__ inline void store4_bf16(bf16* dst, const f32x16& acc, int g, float mul) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  bf16x4 v;
#pragma unroll
  for (int x = 0; x < 4; ++x) v[x] = (bf16)(acc[4 * g + x] * mul);
  *reinterpret_cast<bf16x4*>(dst) = v;
}

// Stage rows [0, 128) x HD of one head into LDS row-major (zero beyond n).
template <int HD, bool NHWC>
__device__ inline void stage_rows(const bf16* __restrict__ src, const Geo& g, const WinTokens<NHWC>& wt, int n,
                                  int hoff, bf16* lds) {
  constexpr int kCpr = HD / 8;
  for (int idx = threadIdx.x; idx < kWinMax * kCpr; idx += kWinThreads) {
    const int row = idx / kCpr;
    const int ch = idx - row * kCpr;
    uint4 raw = make_uint4(0, 0, 0, 0);
    if (row < n) raw = *reinterpret_cast<const uint4*>(src + wt.tok(g, row) * g.C + hoff + ch * 8);
    *reinterpret_cast<uint4*>(lds + row * (HD + 8) + ch * 8) = raw;
  }
}

// Wave `wave` writes the transpose of rows [32*wave, 32*wave+32) of a
// row-major LDS tile (stride HD+8) into dst[e][row] (stride 128+8).
template <int HD>
__device__ inline void transpose_rows_to_lds(const bf16* rows, bf16* dst, int wave) {
  const int lane = threadIdx.x & 63;
  const int h = lane >> 5, col = lane & 31;
  const bf16x8 i0 = ident_op<false>(0), i1 = ident_op<false>(1);
#pragma unroll
  for (int eb = 0; eb < HD / 32; ++eb) {
    const bf16* r = rows + (32 * wave + col) * (HD + 8) + 32 * eb + 8 * h;
    const bf16x8 a0 = *reinterpret_cast<const bf16x8*>(r);
    const bf16x8 a1 = *reinterpret_cast<const bf16x8*>(r + 16);
    const f32x16 t = mfma_transpose(a0, a1, i0, i1);
    // lane holds column e = 32eb + col, rows 32*wave + acc_row(r, h)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4)
      store4_bf16(dst + (32 * eb + col) * (kWinMax + 8) + 32 * wave + 8 * g4 + 4 * h, t, g4, 1.0f);
  }
}

// Operand of 8 keys in pi order from a transposed LDS row.
__device__ inline bf16x8 lds_perm_op(const bf16* row, int h) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  const bf16x4 lo = *reinterpret_cast<const bf16x4*>(row + 4 * h);
  const bf16x4 hi = *reinterpret_cast<const bf16x4*>(row + 8 + 4 * h);
  bf16x8 o;
#pragma unroll
  for (int s = 0; s < 4; ++s) { o[s] = lo[s]; o[4 + s] = hi[s]; }
  return o;
}

__device__ inline bf16x8 pack_bf16(const f32x16& acc, int r0) {
  bf16x8 o;
#pragma unroll
  for (int s = 0; s < 8; ++s) o[s] = (bf16)acc[r0 + s];
  return o;
}

// True when some pair of the window must be excluded: a wrap label inside
// the window or padding slots in its last 32-token block.
__device__ inline bool window_needs_mask(const Geo& g, int wi, int wj, int n) {
  return window_has_labels(g, wi, wj) || (n & 31) != 0;
}

// The same for the backward, whose rotation always covers all four 32-key
// blocks: the padding keys past n also need excluding whenever the window
// is shorter than wh rows, because the bias-gradient flush keeps every key
// whose row (key index / width) lies inside the window height, and padding
// keys of a short window do.  (In a full-height window they sit at row wh
// or beyond and the flush drops them.)
__device__ inline bool window_needs_mask_bwd(const Geo& g, int wi, int wj, int n) {
  return window_needs_mask(g, wi, wj, n) || (n < kWinMax && win_rows(g, wi) < g.wh);
}

// Map a linear block index to a work index so that consecutive work items
// run on the same XCD (blocks are dealt to the 8 XCDs round-robin).
__device__ inline int xcd_work(int bid, int nblocks) {
  if (nblocks % 8 != 0) return bid;
  return (bid % 8) * (nblocks / 8) + bid / 8;
}

// ---------------------------------------------------------------------------
// Forward: one workgroup per (image, window, head); wave w owns queries
// [32w, 32w+32).  Grid B * nwin * heads, head fastest.
// ---------------------------------------------------------------------------
template <int HD, bool QUAD, bool NHWC>
__global__ __launch_bounds__(kWinThreads) void fwd_win_kernel(
    const bf16* __restrict__ q, const bf16* __restrict__ k, const bf16* __restrict__ v,
    const float* __restrict__ table, bf16* __restrict__ o, float* __restrict__ lse, Geo g,
    float scale_log2) {
  extern __shared__ __align__(16) char smem[];
  bf16* ks = reinterpret_cast<bf16*>(smem);                       // [128][HD+8]
  bf16* vts = ks + kWinMax * (HD + 8);                            // [HD][128+8]
  int* kinfo = reinterpret_cast<int*>(vts + HD * (kWinMax + 8));  // [128]
  float* tab = reinterpret_cast<float*>(kinfo + kWinMax);         // [ntab+4]

  int work = xcd_work(blockIdx.x, gridDim.x);
  const int h = work % g.heads; work /= g.heads;
  const int w = work % g.nwin;
  const int b = work / g.nwin;
  const int wi = w / g.Mw, wj = w - (w / g.Mw) * g.Mw;
  const int cols = win_cols(g, wj);
  const int n = win_rows(g, wi) * cols;
  const int nkb = (n + 31) >> 5;
  const WinTokens<NHWC> wt(g, b, wi, wj);
  const int hoff = h * HD;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, col = lane & 31;

  // bias table of head h times sqrt(hd), stored in reverse bin order so that
  // consecutive keys of a window row read consecutive addresses; four -inf
  // entries after it serve excluded pairs
  const float bscale = sqrtf((float)HD);
  for (int x = threadIdx.x; x < g.ntab + 4; x += kWinThreads) tab[x] = table_entry(g, table, h, x, bscale);
  if (threadIdx.x < kWinMax) kinfo[threadIdx.x] = win_token_info(g, wi, wj, cols, threadIdx.x, n);
  stage_rows<HD>(k, g, wt, n, hoff, ks);
  // V^T through LDS: stage V rows into the vts area's tail is not possible
  // (different shapes), so each wave transposes its 32 rows straight from
  // memory.
  if (wave < nkb) {
    const bf16x8 i0 = ident_op<false>(0), i1 = ident_op<false>(1);
    const int row = 32 * wave + col;
#pragma unroll
    for (int eb = 0; eb < HD / 32; ++eb) {
      bf16x8 a0 = zero8(), a1 = zero8();
      if (row < n) {
        const bf16* p = v + wt.tok(g, row) * g.C + hoff + 32 * eb + 8 * half;
        a0 = *reinterpret_cast<const bf16x8*>(p);
        a1 = *reinterpret_cast<const bf16x8*>(p + 16);
      }
      const f32x16 t = mfma_transpose(a0, a1, i0, i1);
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4)
        store4_bf16(vts + (32 * eb + col) * (kWinMax + 8) + 32 * wave + 8 * g4 + 4 * half, t, g4, 1.0f);
    }
  }
  lds_barrier();
  if (wave >= nkb) return;

  const int qi = 32 * wave + col;
  const bool qvalid = qi < n;
  const int qinf = kinfo[qvalid ? qi : 0];
  const int qlab = qinf >> 24;
  // reversed bin of (q, k) = qrev + koff(k)
  const int qrev = table_qrev(g, qinf);
  bf16x8 qop[HD / 16];
#pragma unroll
  for (int c = 0; c < HD / 16; ++c)
    qop[c] = qvalid ? *reinterpret_cast<const bf16x8*>(q + wt.tok(g, qi) * g.C + hoff + 16 * c + 8 * half)
                    : zero8();

  // raw scores with the bias folded into the accumulator: s = QK^T + bias*sqrt(hd)
  f32x16 s[4];
  const bool mask = window_needs_mask(g, wi, wj, n);
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    if (kb < nkb) {
      s[kb] = mask ? bias_init<QUAD, true>(kinfo, tab, kb, half, qrev, qlab, g.ntab)
                   : bias_init<QUAD, false>(kinfo, tab, kb, half, qrev, qlab, g.ntab);
#pragma unroll
      for (int c = 0; c < HD / 16; ++c)
        mma16(s[kb], *reinterpret_cast<const bf16x8*>(ks + (32 * kb + col) * (HD + 8) + 16 * c + 8 * half),
              qop[c]);
    }
  }
  float mr = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
    if (kb < nkb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mr = fmaxf(mr, s[kb][r]);
  mr = halves_max(mr);
  const float m = mr * scale_log2;            // row max, log2 domain
  float l = 0.0f;
  f32x16 oacc[HD / 32];
#pragma unroll
  for (int eb = 0; eb < HD / 32; ++eb) oacc[eb] = f32x16{};
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    if (kb < nkb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(s[kb][r] * scale_log2 - m);
        s[kb][r] = p;
        l += p;
      }
#pragma unroll
      for (int eb = 0; eb < HD / 32; ++eb)
#pragma unroll
        for (int c = 0; c < 2; ++c)
          mma16(oacc[eb], lds_perm_op(vts + (32 * eb + col) * (kWinMax + 8) + 32 * kb + 16 * c, half),
                pack_bf16(s[kb], 8 * c));
    }
  }
  l = halves_sum(l);
  if (!qvalid) return;
  const float inv = 1.0f / l;
  bf16* orow = o + wt.tok(g, qi) * g.C + hoff;
#pragma unroll
  for (int eb = 0; eb < HD / 32; ++eb)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) store4_bf16(orow + 32 * eb + 8 * g4 + 4 * half, oacc[eb], g4, inv);
  if (half == 0) lse[wt.lse_at(g, h, qi)] = (m + __log2f(l)) * kLn2;
}

// ---------------------------------------------------------------------------
// Forward for head_dim 32 and an even head count: one workgroup of 8 waves
// per (head pair, run of consecutive windows), two resident per CU.  Each
// window's rows are loaded into registers while the previous window
// computes (126 registers, still four waves per SIMD; -4 % against loading
// at the top of each window).  Global memory is touched only in
// row-contiguous 128-byte segments (8 lanes per token row): Q, K and V are
// staged through LDS (V row-major, read transposed by the LDS transpose
// read) and O goes back through LDS.  Wave w handles head 2*hp + (w >> 2)
// and queries [32*(w&3), 32*(w&3)+32).
// ---------------------------------------------------------------------------
constexpr int kPairThreads = 512;

// Rows of one window and head pair on their way from HBM to LDS: thread t
// holds 16-byte chunks t and t+512 (row = chunk / 8) of K, Q and V.
struct PairRows {
  uint4 k[2], q[2], v[2];
};

template <bool NHWC>
__device__ __forceinline__ void pair_load_rows(PairRows& r, const Geo& g, int wl, int64_t cbase,
                                               const bf16* __restrict__ q, const bf16* __restrict__ k,
                                               const bf16* __restrict__ v) {
  const int b = wl / g.nwin;
  const int w = wl - b * g.nwin;
  const int wi = w / g.Mw, wj = w - (w / g.Mw) * g.Mw;
  const int n = win_rows(g, wi) * win_cols(g, wj);
  const WinTokens<NHWC> wt(g, b, wi, wj);
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int idx = threadIdx.x + u * kPairThreads;
    const int row = idx >> 3, ch = idx & 7;
    r.k[u] = r.q[u] = r.v[u] = make_uint4(0, 0, 0, 0);
    if (row < n) {
      const int64_t off = wt.tok(g, row) * g.C + cbase + ch * 8;
      r.k[u] = *reinterpret_cast<const uint4*>(k + off);
      r.q[u] = *reinterpret_cast<const uint4*>(q + off);
      r.v[u] = *reinterpret_cast<const uint4*>(v + off);
    }
  }
}

template <bool QUAD, bool NHWC>
__global__ __launch_bounds__(kPairThreads, 4) void fwd_win_pair_kernel(
    const bf16* __restrict__ q, const bf16* __restrict__ k, const bf16* __restrict__ v,
    const float* __restrict__ table, bf16* __restrict__ o, float* __restrict__ lse, Geo g,
    int per_slice, float scale_log2) {
  constexpr int HD = 32;
  // V stays row-major (64-byte rows): its transposed operands come through
  // the LDS transpose read, 4 rows x 64 bytes of two lane groups in
  // distinct banks
  constexpr int KS = HD + 8, VH = kWinMax * HD;
  extern __shared__ __align__(16) char smem[];
  bf16* ks = reinterpret_cast<bf16*>(smem);                        // [2][128][KS] K rows
  bf16* qs = ks + 2 * kWinMax * KS;                                // [2][128][KS] Q rows, then O
  bf16* vrs = qs + 2 * kWinMax * KS;                               // [2][128][HD] V rows
  int* kinfo = reinterpret_cast<int*>(vrs + 2 * VH);               // [128]
  float* tab = reinterpret_cast<float*>(kinfo + kWinMax);          // [2][ntab+4]

  const int hpairs = g.heads >> 1;
  const int work = xcd_work(blockIdx.x, gridDim.x);
  const int slice = work / hpairs;
  const int hp = work - slice * hpairs;
  const int64_t cbase = (int64_t)2 * hp * HD;          // first channel of the pair
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int hs = wave >> 2, qb = wave & 3;
  const int h = 2 * hp + hs;
  const int qi = 32 * qb + col;
  const bf16* ksh = ks + hs * kWinMax * KS;
  const bf16* vth = vrs + hs * VH;
  const float* tabh = tab + hs * (g.ntab + 4);

  // bias tables of the pair times sqrt(hd), reversed, then four -inf
  const float bscale = sqrtf((float)HD);
  for (int x = threadIdx.x; x < 2 * (g.ntab + 4); x += kPairThreads) {
    const int t = x / (g.ntab + 4), y = x - t * (g.ntab + 4);
    tab[x] = table_entry(g, table, 2 * hp + t, y, bscale);
  }

  const int total = g.B * g.nwin;
  const int wbeg = slice * per_slice;
  const int wend = min(total, wbeg + per_slice);
  PairRows rows;
  for (int wl = wbeg; wl < wend; ++wl) {
    const int b = wl / g.nwin;
    const int w = wl - b * g.nwin;
    const int wi = w / g.Mw, wj = w - (w / g.Mw) * g.Mw;
    const int cols = win_cols(g, wj);
    const int n = win_rows(g, wi) * cols;
    const int nkb = (n + 31) >> 5;
    const WinTokens<NHWC> wt(g, b, wi, wj);
    const bool qvalid = qi < n;

    if (wl == wbeg) pair_load_rows<NHWC>(rows, g, wl, cbase, q, k, v);
    lds_barrier();   // the previous window is done with LDS
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int idx = threadIdx.x + u * kPairThreads;
      const int row = idx >> 3, ch = idx & 7;
      const int t = ch >> 2, e0 = (ch & 3) * 8;
      *reinterpret_cast<uint4*>(ks + (t * kWinMax + row) * KS + e0) = rows.k[u];
      *reinterpret_cast<uint4*>(qs + (t * kWinMax + row) * KS + e0) = rows.q[u];
      *reinterpret_cast<uint4*>(vrs + t * VH + row * HD + e0) = rows.v[u];
    }
    if (threadIdx.x < kWinMax) kinfo[threadIdx.x] = win_token_info(g, wi, wj, cols, threadIdx.x, n);
    lds_barrier();
    if (wl + 1 < wend) pair_load_rows<NHWC>(rows, g, wl + 1, cbase, q, k, v);   // next window

    // Softmax over the two halves of the window's keys in turn (running
    // max and sum; a half with no allowed key for a query leaves it as it
    // was), so that only 32 score registers are live.
    const bool active = qb < nkb;
    f32x16 oacc = f32x16{};
    float m = -INFINITY, l = 0.0f;
    if (active) {
      bf16x8 qop[2];
#pragma unroll
      for (int c = 0; c < 2; ++c)
        qop[c] = *reinterpret_cast<const bf16x8*>(qs + (hs * kWinMax + qi) * KS + 16 * c + 8 * half);
      const int qinf = kinfo[qvalid ? qi : 0];
      const int qlab = qinf >> 24;
      const int qrev = table_qrev(g, qinf);
      const bool mask = window_needs_mask(g, wi, wj, n);
#pragma unroll
      for (int hb = 0; hb < 2; ++hb) {
        if (2 * hb < nkb) {
          f32x16 s[2];
          float mr = -INFINITY;
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const int kb = 2 * hb + j;
            if (kb < nkb) {
              s[j] = mask ? bias_init<QUAD, true>(kinfo, tabh, kb, half, qrev, qlab, g.ntab)
                          : bias_init<QUAD, false>(kinfo, tabh, kb, half, qrev, qlab, g.ntab);
#pragma unroll
              for (int c = 0; c < 2; ++c)
                mma16(s[j], *reinterpret_cast<const bf16x8*>(ksh + (32 * kb + col) * KS + 16 * c + 8 * half),
                      qop[c]);
#pragma unroll
              for (int r = 0; r < 16; ++r) mr = fmaxf(mr, s[j][r]);
            }
          }
          mr = halves_max(mr);
          const float mnew = fmaxf(m, mr * scale_log2);
          const float mref = mnew == -INFINITY ? 0.0f : mnew;   // nothing allowed yet
          if (hb > 0) {   // the first half starts from l = 0, O = 0
            const float alpha = __builtin_amdgcn_exp2f(m - mref);
            l *= alpha;
#pragma unroll
            for (int r = 0; r < 16; ++r) oacc[r] *= alpha;
          }
          m = mnew;
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const int kb = 2 * hb + j;
            if (kb < nkb) {
#pragma unroll
              for (int r = 0; r < 16; ++r) {
                const float p = __builtin_amdgcn_exp2f(s[j][r] * scale_log2 - mref);
                s[j][r] = p;
                l += p;
              }
#pragma unroll
              for (int c = 0; c < 2; ++c)
                mma16(oacc, lds_tr_op<bf16, HD>(vth, kb, c, 0, lane), pack_bf16(s[j], 8 * c));
            }
          }
        }
      }
      l = halves_sum(l);
    }
    lds_barrier();   // every wave has read its Q rows; qs now takes O
    if (active) {
      const float inv = 1.0f / l;
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4)
        store4_bf16(qs + (hs * kWinMax + qi) * KS + 8 * g4 + 4 * half, oacc, g4, inv);
      if (qvalid && half == 0) lse[wt.lse_at(g, h, qi)] = (m + __log2f(l)) * kLn2;
    }
    lds_barrier();
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int idx = threadIdx.x + u * kPairThreads;
      const int row = idx >> 3, ch = idx & 7;
      if (row < n) {
        const int t = ch >> 2, e0 = (ch & 3) * 8;
        // streaming store: O is not read again by this path (the backward
        // recomputes P), so it should not displace the inputs in the caches
        typedef unsigned int u32x4n __attribute__((ext_vector_type(4)));
        __builtin_nontemporal_store(*reinterpret_cast<const u32x4n*>(qs + (t * kWinMax + row) * KS + e0),
                                    reinterpret_cast<u32x4n*>(o + wt.tok(g, row) * g.C + cbase + ch * 8));
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Backward (head_dim 32): one workgroup of 4 waves per (head, run of
// consecutive windows), two workgroups resident per CU so that one's memory
// phase overlaps the other's matrix work.  Per window, wave w owns queries
// [32w, 32w+32) for P, dP, D, dS and dQ; the four waves then rotate over the
// key blocks to sum dV and dK in LDS.
// ---------------------------------------------------------------------------
constexpr int kBwdHD = 32;
constexpr int kBwdKS = kBwdHD + 8;     // LDS row stride (bf16) of K, V, Q, dO rows
constexpr int kBwdRS = kWinMax + 4;    // LDS row stride (fp32) of the dV, dK sums
constexpr int kBwdRed = 32 * kBwdRS + 16;   // floats of one sum array

// Row of channel e in the dV/dK sum arrays: channels 16..31 sit 16 words
// further, so that the output stage's transposing reads (16 token rows of
// four 8-channel groups per instruction) fall in distinct LDS banks; the
// rotation's 16-byte accesses of 16 channels stay in distinct banks too.
__device__ __forceinline__ int red_row(int e) { return e * kBwdRS + (e >> 4) * 16; }
constexpr int kBwdCPR = kBwdHD / 8;    // 16-byte chunks per token row of one head

// Token row of 16-byte chunk idx (chunk idx % 4 of its row) in the
// row-contiguous staging of one head: the 16 lanes of a group take rows
// r, r+4, r+8, r+12 of a 16-row band, whose 64-byte LDS row segments
// (80-byte row stride) then fall in distinct banks.
__device__ __forceinline__ int bwd_stage_row(int idx) {
  const int blk = idx >> 4;
  return ((blk >> 2) << 4) + (blk & 3) + 4 * ((idx >> 2) & 3);
}

// Per-lane 0/1 factors of the bias-gradient fold for the window width cols
// (a multiple of 4 that divides 32, so window rows never straddle a 32-lane
// half): cq is the lane's query column.
struct FoldMask {
  float next;     // lane l+1 holds the next query of the same window row
  float b0, b1, b2;
};

__device__ __forceinline__ FoldMask fold_mask(int cq, int cols) {
  FoldMask m;
  m.next = cq < cols - 1 ? 1.0f : 0.0f;
  m.b0 = cq < 3 ? 1.0f : 0.0f;
  m.b1 = (cq == 1 || cq == 2) ? 1.0f : 0.0f;
  m.b2 = cq == 2 ? 1.0f : 0.0f;
  return m;
}

// Per-wave state of the backward for one window.
struct BwdWave {
  const bf16* ks;       // K rows in LDS [128][KS]
  const bf16* vs;       // V rows [128][KS]
  const int* kinfo;     // key words of the window
  const float* tab;     // bias table times sqrt(hd), reversed, then -inf
  float* redv;          // dV partial sums [HD][RS]
  float* redk;          // dK partial sums [HD][RS]
  const bf16* qr;       // Q rows [128][HD] (transposed operands read from here)
  const bf16* dr;       // dO rows [128][HD]
  bf16x8 qop[2], dop[2];  // Q and dO of the wave's 32 queries (row operands)
  float D, lse2, scale_log2;
  FoldMask fold;
  int qrev, qlab, ntab, col, half, qw;
};

// dS summed along the bias diagonals of one register group: registers
// 4g..4g+3 hold four consecutive keys k..k+3 of one window row, so (query q,
// key k+x) and (q+1, k+x+1) share a bin when q+1 is in q's window row.  A
// chain towards lower lanes leaves in lane q the sum of the bin of (q, k);
// the pairs it cannot reach (query column cq < x) have the bins of
// (q', k+3) for the three first queries q' of the row, summed into `b` there.
// Group g4 updates a[g4] and b[g4].
__device__ __forceinline__ void fold_diag(const f32x16& ds, int g4, const FoldMask& m, f32x4& a,
                                          f32x4& b) {
  float f = ds[4 * g4 + 3];
  f = ds[4 * g4 + 2] + m.next * dpp_lane<kDppNext>(f);
  f = ds[4 * g4 + 1] + m.next * dpp_lane<kDppNext>(f);
  a[g4] += ds[4 * g4] + m.next * dpp_lane<kDppNext>(f);
  b[g4] += m.b0 * ds[4 * g4 + 3];
  b[g4] += m.b1 * dpp_lane<kDppPrev1>(ds[4 * g4 + 2]);
  b[g4] += m.b2 * dpp_lane<kDppPrev2>(ds[4 * g4 + 1]);
}

// P of key block KB for the wave's queries (lane = query, registers = keys):
// bias in the accumulator, S = K Q^T on the matrix cores, exp2 against the
// saved log-sum-exp (+inf for padding queries, so their P is 0).
template <int KB, bool QUAD, bool MASK>
__device__ __forceinline__ f32x16 bwd_p(const BwdWave& st) {
  f32x16 p = bias_init<QUAD, MASK>(st.kinfo, st.tab, KB, st.half, st.qrev, st.qlab, st.ntab);
#pragma unroll
  for (int c = 0; c < 2; ++c)
    mma16(p, *reinterpret_cast<const bf16x8*>(st.ks + (32 * KB + st.col) * kBwdKS + 16 * c + 8 * st.half),
          st.qop[c]);
#pragma unroll
  for (int r = 0; r < 16; ++r) p[r] = __builtin_amdgcn_exp2f(p[r] * st.scale_log2 - st.lse2);
  return p;
}

// dP of key block KB (lane = query, registers = keys), plus `init` (the
// accumulator's starting value: 0, or -D so that dP - D comes out directly).
template <int KB>
__device__ __forceinline__ f32x16 bwd_dp(const BwdWave& st, float init) {
  f32x16 dp;
#pragma unroll
  for (int r = 0; r < 16; ++r) dp[r] = init;
#pragma unroll
  for (int c = 0; c < 2; ++c)
    mma16(dp, *reinterpret_cast<const bf16x8*>(st.vs + (32 * KB + st.col) * kBwdKS + 16 * c + 8 * st.half),
          st.dop[c]);
  return dp;
}

// One rotation step: key block KB.  P and dP are recomputed (so that P does
// not occupy 64 registers across the steps; steps 0, 1 and 2 take them
// from the D pass), dS = P (dP - D) goes into the bias accumulators and into
// dQ += dS K (K^T operands by the LDS transpose read of the K rows); P^T and
// dS^T (by matrix-core transpose) times dO and Q give the block's dV and dK
// partials, which are added to the running sums in LDS through the
// accumulator input.  Step T = 0 starts the sums.
template <int KB, int T>
__device__ __forceinline__ void bwd_step_tail(const BwdWave& st, const f32x16& p, const f32x16& ds, f32x4& dta,
                                              f32x4& dtb, f32x16& dqacc) {
  bf16x8 pb0, pb1, db0, db1;
#pragma unroll
  for (int g4 = 0; g4 < 4; ++g4) fold_diag(ds, g4, st.fold, dta, dtb);
  pb0 = pack_bf16(p, 0); pb1 = pack_bf16(p, 8);
  db0 = pack_bf16(ds, 0); db1 = pack_bf16(ds, 8);
  const int lane = threadIdx.x & 63;
  mma16(dqacc, lds_tr_op<bf16, kBwdKS>(st.ks, KB, 0, 0, lane), db0);
  mma16(dqacc, lds_tr_op<bf16, kBwdKS>(st.ks, KB, 1, 0, lane), db1);
#pragma unroll
  for (int which = 0; which < 2; ++which) {
    const bf16x8 ip0 = ident_op<true>(0), ip1 = ident_op<true>(1);
    const f32x16 tr = which == 0 ? mfma_transpose(pb0, pb1, ip0, ip1) : mfma_transpose(db0, db1, ip0, ip1);
    float* red = which == 0 ? st.redv : st.redk;
    f32x16 part;
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const f32x4 a = T > 0 ? *reinterpret_cast<const f32x4*>(red + red_row(st.col) + 32 * KB + 8 * g4 + 4 * st.half)
                            : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int x = 0; x < 4; ++x) part[4 * g4 + x] = a[x];
    }
    // dO or Q of the wave's queries with lane = channel, by the LDS
    // transpose read of their rows
    const bf16* rows = which == 0 ? st.dr : st.qr;
    mma16(part, pack_bf16(tr, 0), lds_tr_op<bf16, kBwdHD>(rows, st.qw, 0, 0, lane));
    mma16(part, pack_bf16(tr, 8), lds_tr_op<bf16, kBwdHD>(rows, st.qw, 1, 0, lane));
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4)
      *reinterpret_cast<f32x4*>(red + red_row(st.col) + 32 * KB + 8 * g4 + 4 * st.half) =
          f32x4{part[4 * g4], part[4 * g4 + 1], part[4 * g4 + 2], part[4 * g4 + 3]};
  }
}

template <int KB, int T, bool QUAD, bool MASK>
__device__ __forceinline__ void bwd_step(const BwdWave& st, f32x4& dta, f32x4& dtb, f32x16& dqacc) {
  const f32x16 p = bwd_p<KB, QUAD, MASK>(st);
  f32x16 ds = bwd_dp<KB>(st, -st.D);
#pragma unroll
  for (int r = 0; r < 16; ++r) ds[r] *= p[r];
  bwd_step_tail<KB, T>(st, p, ds, dta, dtb, dqacc);
}

// The wave with query block W: pass 1 forms D = sum_k P dP over key blocks
// W+3, W+2, W+1, W (mod 4), the last three P and dP kept for steps 2, 1
// and 0; then
// the four steps over key blocks W, W+1, W+2, W+3, so that at every step
// each block is touched by exactly one wave; a barrier ends each step, so
// the order of additions into every block is fixed.
template <int W, bool QUAD, bool MASK>
__device__ __forceinline__ void bwd_rotation(BwdWave& st, f32x4 (&dta)[4], f32x4 (&dtb)[4], f32x16& dqacc) {
  float dsum = 0.0f;
#define TERRA_DSUM(KB)                                                          \
  {                                                                             \
    const f32x16 pk = bwd_p<KB, QUAD, MASK>(st);                                \
    const f32x16 dk = bwd_dp<KB>(st, 0.0f);                                     \
    _Pragma("unroll") for (int r = 0; r < 16; ++r) dsum += pk[r] * dk[r];       \
  }
  TERRA_DSUM((W + 3) & 3)
#undef TERRA_DSUM
  const f32x16 p2 = bwd_p<(W + 2) & 3, QUAD, MASK>(st);
  f32x16 ds2 = bwd_dp<(W + 2) & 3>(st, 0.0f);
#pragma unroll
  for (int r = 0; r < 16; ++r) dsum += p2[r] * ds2[r];
  const f32x16 p1 = bwd_p<(W + 1) & 3, QUAD, MASK>(st);
  f32x16 ds1 = bwd_dp<(W + 1) & 3>(st, 0.0f);
#pragma unroll
  for (int r = 0; r < 16; ++r) dsum += p1[r] * ds1[r];
  const f32x16 p0 = bwd_p<W, QUAD, MASK>(st);
  f32x16 ds0 = bwd_dp<W>(st, 0.0f);
#pragma unroll
  for (int r = 0; r < 16; ++r) dsum += p0[r] * ds0[r];
  st.D = halves_sum(dsum);
#pragma unroll
  for (int r = 0; r < 16; ++r) ds0[r] = p0[r] * (ds0[r] - st.D);
#pragma unroll
  for (int r = 0; r < 16; ++r) ds1[r] = p1[r] * (ds1[r] - st.D);
#pragma unroll
  for (int r = 0; r < 16; ++r) ds2[r] = p2[r] * (ds2[r] - st.D);
  bwd_step_tail<W, 0>(st, p0, ds0, dta[W], dtb[W], dqacc);
  lds_barrier();
  bwd_step_tail<(W + 1) & 3, 1>(st, p1, ds1, dta[(W + 1) & 3], dtb[(W + 1) & 3], dqacc);
  lds_barrier();
  bwd_step_tail<(W + 2) & 3, 2>(st, p2, ds2, dta[(W + 2) & 3], dtb[(W + 2) & 3], dqacc);
  lds_barrier();
  bwd_step<(W + 3) & 3, 3, QUAD, MASK>(st, dta[(W + 3) & 3], dtb[(W + 3) & 3], dqacc);
  lds_barrier();
}

template <bool QUAD, bool MASK>
__device__ __forceinline__ void bwd_window_body(BwdWave& st, int qw, f32x4 (&dta)[4], f32x4 (&dtb)[4],
                                                f32x16& dqacc) {
  switch (qw) {
    case 0: bwd_rotation<0, QUAD, MASK>(st, dta, dtb, dqacc); break;
    case 1: bwd_rotation<1, QUAD, MASK>(st, dta, dtb, dqacc); break;
    case 2: bwd_rotation<2, QUAD, MASK>(st, dta, dtb, dqacc); break;
    default: bwd_rotation<3, QUAD, MASK>(st, dta, dtb, dqacc); break;
  }
}

// Rows of one window on their way from HBM to LDS: thread t holds 16-byte
// chunks t and t+256 (row bwd_stage_row(chunk)) of K, V, Q and dO, and the
// log-sum-exp (log2 units) of its wave's query.
struct BwdRows {
  uint4 k[2], v[2], q[2], d[2];
  float lse2;
};

template <bool NHWC>
__device__ __forceinline__ void bwd_load_rows(BwdRows& r, const Geo& g, int wl, int h, int qi,
                                              const bf16* __restrict__ q, const bf16* __restrict__ k,
                                              const bf16* __restrict__ v, const bf16* __restrict__ dout,
                                              const float* __restrict__ lse) {
  const int b = wl / g.nwin;
  const int w = wl - b * g.nwin;
  const int wi = w / g.Mw, wj = w - (w / g.Mw) * g.Mw;
  const int n = win_rows(g, wi) * win_cols(g, wj);
  const WinTokens<NHWC> wt(g, b, wi, wj);
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int idx = threadIdx.x + u * kWinThreads;
    const int row = bwd_stage_row(idx), ch = idx % kBwdCPR;
    r.k[u] = r.v[u] = r.q[u] = r.d[u] = make_uint4(0, 0, 0, 0);
    if (row < n) {
      const int64_t off = wt.tok(g, row) * g.C + h * kBwdHD + ch * 8;
      r.k[u] = *reinterpret_cast<const uint4*>(k + off);
      r.v[u] = *reinterpret_cast<const uint4*>(v + off);
      r.q[u] = *reinterpret_cast<const uint4*>(q + off);
      r.d[u] = *reinterpret_cast<const uint4*>(dout + off);
    }
  }
  r.lse2 = qi < n ? lse[wt.lse_at(g, h, qi)] * kLog2e : INFINITY;
}

// Backward, head_dim 32, window widths in {4, 8, 16, 32}.  K, V, Q and dO
// arrive with row-contiguous loads (the other workgroup resident on the CU
// computes meanwhile; loading one window ahead measured slower) and stay in
// LDS for the whole window (80 KB in all, two workgroups per CU).  dQ, dK
// and dV leave with row-contiguous stores.  The bias-gradient sums of every
// register run over windows of equal width and are flushed to per-wave LDS
// bins when the width changes (a register holds the same query/key slot
// pair, hence the same bin, in every such window).
template <bool QUAD, bool NHWC>
__global__ __launch_bounds__(kWinThreads, 2) void bwd_win_kernel(
    const bf16* __restrict__ q, const bf16* __restrict__ k, const bf16* __restrict__ v,
    const bf16* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ table,
    bf16* __restrict__ dq, bf16* __restrict__ dk, bf16* __restrict__ dv,
    float* __restrict__ partial, Geo g, int nslice, int per_slice, float scale_log2, float scale) {
  constexpr int HD = kBwdHD;
  constexpr int KS = kBwdKS;
  extern __shared__ __align__(16) char smem[];
  bf16* ks = reinterpret_cast<bf16*>(smem);                     // [128][KS] K rows, then dQ
  bf16* vs = ks + kWinMax * KS;                                 // [128][KS] V rows
  bf16* qr = vs + kWinMax * KS;                                 // [128][HD] Q rows
  bf16* dr = qr + kWinMax * HD;                                 // [128][HD] dO rows
  float* redv = reinterpret_cast<float*>(dr + kWinMax * HD);    // [HD][RS] dV sums
  float* redk = redv + kBwdRed;                                 // [HD][RS] dK sums
  int* kinfo = reinterpret_cast<int*>(redk + kBwdRed);          // [128]
  float* tab = reinterpret_cast<float*>(kinfo + kWinMax);       // [ntab+4]
  float* bins = tab + (g.ntab + 4);                             // [4][nbins], reversed

  const int work = xcd_work(blockIdx.x, gridDim.x);
  const int slice = work / g.heads;
  const int h = work - slice * g.heads;
  const int lane = threadIdx.x & 63;
  const int qw = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int half = lane >> 5, col = lane & 31;
  const int qi = 32 * qw + col;
  float* mybins = bins + qw * g.nbins;

  for (int x = threadIdx.x; x < 4 * g.nbins; x += kWinThreads) bins[x] = 0.0f;
  for (int x = threadIdx.x; x < g.ntab + 4; x += kWinThreads)
    tab[x] = table_entry(g, table, h, x, sqrtf((float)HD));

  f32x4 dta[4], dtb[4];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) dta[kb] = dtb[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
  int acc_cols = 0;
  // Register (kb, g4) of lane q holds, in dta, the bin of (q, k) with k the
  // group's first key, and in dtb (query columns 0..2 only) the bin of
  // (q, k+3).  The two lane halves flush with separate instructions: within
  // one half the lanes hold distinct queries of the same key, hence distinct
  // bins, so the additions are plain read-modify-writes in program order (an
  // LDS float atomic costs about three clocks per lane).
#define TERRA_FLUSH_DT(cw)                                                              \
  {                                                                                     \
    /* widths are powers of two here (4, 8, 16 or 32): rows and columns by shifts, */   \
    /* so that nothing of the flush is kept live across the window loop */             \
    const int lw = __builtin_ctz((unsigned)(cw));                                       \
    const int aq = qi >> lw, cq = qi & ((cw) - 1);                                      \
    _Pragma("unroll 1") for (int hh = 0; hh < 2; ++hh) {                                \
      if (half == hh) {                                                                 \
        _Pragma("unroll") for (int kb = 0; kb < 4; ++kb)                                \
        _Pragma("unroll") for (int g4 = 0; g4 < 4; ++g4) {                              \
          const int kk = 32 * kb + 8 * g4 + 4 * hh;                                     \
          const int ak = kk >> lw, ck = kk & ((cw) - 1);                                \
          if (aq < g.wh && ak < g.wh) {                                                 \
            const int bin = g.nbins - 1 - ((aq - ak + g.wh - 1) * g.bstride + (cq - ck + g.ww - 1)); \
            mybins[bin] += dta[kb][g4];                                                 \
            if (cq < 3) mybins[bin + 3] += dtb[kb][g4];                                 \
          }                                                                             \
        }                                                                               \
      }                                                                                 \
      __builtin_amdgcn_wave_barrier();                                                  \
    }                                                                                   \
    _Pragma("unroll") for (int kb = 0; kb < 4; ++kb) dta[kb] = dtb[kb] = f32x4{0.f, 0.f, 0.f, 0.f}; \
  }

  const int total = g.B * g.nwin;
  const int wbeg = slice * per_slice;
  const int wend = min(total, wbeg + per_slice);
  BwdRows rows;
  for (int wl = wbeg; wl < wend; ++wl) {
    const int b = wl / g.nwin;
    const int w = wl - b * g.nwin;
    const int wi = w / g.Mw, wj = w - (w / g.Mw) * g.Mw;
    const int cols = win_cols(g, wj);
    const int n = win_rows(g, wi) * cols;
    const WinTokens<NHWC> wt(g, b, wi, wj);
    if (cols != acc_cols) {          // uniform across the workgroup
      if (acc_cols > 0) TERRA_FLUSH_DT(acc_cols);
      acc_cols = cols;
    }

    bwd_load_rows<NHWC>(rows, g, wl, h, qi, q, k, v, dout, lse);
    lds_barrier();   // the previous window is done with LDS
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int idx = threadIdx.x + u * kWinThreads;
      const int row = bwd_stage_row(idx), c0 = (idx % kBwdCPR) * 8;
      *reinterpret_cast<uint4*>(ks + row * KS + c0) = rows.k[u];
      *reinterpret_cast<uint4*>(vs + row * KS + c0) = rows.v[u];
      *reinterpret_cast<uint4*>(qr + row * HD + c0) = rows.q[u];
      *reinterpret_cast<uint4*>(dr + row * HD + c0) = rows.d[u];
    }
    if (threadIdx.x < kWinMax) kinfo[threadIdx.x] = win_token_info(g, wi, wj, cols, threadIdx.x, n);
    BwdWave st;
    st.lse2 = rows.lse2;
    lds_barrier();

    st.ks = ks;
    st.vs = vs;
    st.kinfo = kinfo;
    st.tab = tab;
    st.redv = redv;
    st.redk = redk;
    st.qr = qr;
    st.dr = dr;
    st.qw = qw;
    st.scale_log2 = scale_log2;
    st.ntab = g.ntab;
    st.col = col;
    st.half = half;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      st.qop[c] = *reinterpret_cast<const bf16x8*>(qr + qi * HD + 16 * c + 8 * half);
      st.dop[c] = *reinterpret_cast<const bf16x8*>(dr + qi * HD + 16 * c + 8 * half);
    }
    const int qinf = qi < n ? kinfo[qi] : 0;
    st.qlab = qinf >> 24;
    st.qrev = table_qrev(g, qinf);
    st.fold = fold_mask(qi % cols, cols);
    f32x16 dqacc = f32x16{};
    if (window_needs_mask_bwd(g, wi, wj, n)) bwd_window_body<QUAD, true>(st, qw, dta, dtb, dqacc);
    else bwd_window_body<QUAD, false>(st, qw, dta, dtb, dqacc);

    // dQ rows of the wave into the K-row area (free after the rotation),
    // then row-contiguous stores of dQ, dV and dK
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) store4_bf16(ks + qi * KS + 8 * g4 + 4 * half, dqacc, g4, scale);
    lds_barrier();
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int idx = threadIdx.x + u * kWinThreads;
      const int row = bwd_stage_row(idx), c0 = (idx % kBwdCPR) * 8;
      if (row < n) {
        const int64_t off = wt.tok(g, row) * g.C + h * HD + c0;
        *reinterpret_cast<uint4*>(dq + off) = *reinterpret_cast<const uint4*>(ks + row * KS + c0);
        bf16x8 a, bb;
#pragma unroll
        for (int x = 0; x < 8; ++x) {
          a[x] = (bf16)redv[red_row(c0 + x) + row];
          bb[x] = (bf16)(redk[red_row(c0 + x) + row] * scale);
        }
        *reinterpret_cast<bf16x8*>(dv + off) = a;
        *reinterpret_cast<bf16x8*>(dk + off) = bb;
      }
    }
  }
  if (acc_cols > 0) TERRA_FLUSH_DT(acc_cols);
#undef TERRA_FLUSH_DT
  lds_barrier();
  for (int y = threadIdx.x; y < g.nbins; y += kWinThreads) {
    const int ry = g.nbins - 1 - y;
    partial[((int64_t)h * nslice + slice) * g.nbins + y] =
        ((bins[ry] + bins[g.nbins + ry]) + bins[2 * g.nbins + ry]) + bins[3 * g.nbins + ry];
  }
}

// ---------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------
bool win_fwd_ok(const Geo& g, bool bf16_) { return bf16_ && g.wh * g.ww <= kWinMax && (g.hd == 32 || g.hd == 64); }
// The backward folds the bias gradient along groups of four keys of one
// window row across lanes, so every window width must be a multiple of 4
// that divides 32 (window rows never straddle a 32-lane half).
static bool fold_width(int w) { return w == 4 || w == 8 || w == 16 || w == 32; }
// Windows of at most 64 tokens go to the generic kernels: this kernel's
// rotation always covers four 32-key blocks, half of them empty for such
// windows (8x8 windows: backward 0.080 ms here, 0.067 ms generic).
bool win_bwd_ok(const Geo& g, bool bf16_) {
  return bf16_ && g.wh * g.ww <= kWinMax && g.wh * g.ww > 64 && g.hd == kBwdHD && fold_width(g.ww) &&
         (g.W % g.ww == 0 || fold_width(g.W % g.ww));
}

// Slices of the window range per head; a pure function of the geometry.
size_t win_bwd_lds(const Geo& g);

// Slices of the window range per head: one round of workgroups over the
// device's CUs, two resident per CU (two waves per SIMD; the LDS plan fits twice in
// 160 KB), so that one workgroup's memory phase overlaps the other's matrix
// work.  A pure function of the geometry.
int win_bwd_nslice(const Geo& g) {
  const int total = g.B * g.nwin;
  const int per_cu = win_bwd_lds(g) * 2 <= 160 * 1024 ? 2 : 1;
  int target = g.cus * per_cu / g.heads;
  if (target > total) target = total;
  if (target < 1) target = 1;
  const int per = (total + target - 1) / target;
  return (total + per - 1) / per;
}

size_t win_fwd_pair_lds(const Geo& g);
size_t win_fwd_lds(const Geo& g) {
  const size_t one = sizeof(bf16) * (kWinMax * (g.hd + 8) + g.hd * (kWinMax + 8)) + 4 * kWinMax +
                     4 * (g.ntab + 4);
  if (g.hd == 32 && g.heads % 2 == 0) {
    const size_t pair = win_fwd_pair_lds(g);
    return pair > one ? pair : one;
  }
  return one;
}
size_t win_bwd_lds(const Geo& g) {
  return sizeof(bf16) * (2 * kWinMax * kBwdKS + 2 * kWinMax * kBwdHD) +
         sizeof(float) * 2 * kBwdRed + 4 * kWinMax + 4 * (g.ntab + 4) + 4 * 4 * g.nbins;
}


template <int HD, bool QUAD, bool NHWC>
static void fwd_win_go(const Geo& g, const void* q, const void* k, const void* v,
                       const float* table, void* o, float* lse, hipStream_t st) {
  const int grid = g.B * g.nwin * g.heads;
  const float sl2 = kLog2e / sqrtf((float)g.hd);
  hipLaunchKernelGGL((fwd_win_kernel<HD, QUAD, NHWC>), dim3(grid), dim3(kWinThreads), win_fwd_lds(g), st,
                     (const bf16*)q, (const bf16*)k, (const bf16*)v, table, (bf16*)o, lse, g, sl2);
}

size_t win_fwd_pair_lds(const Geo& g) {
  return sizeof(bf16) * 2 * (2 * kWinMax * (32 + 8) + kWinMax * 32) + 4 * kWinMax + 4 * 2 * (g.ntab + 4);
}

// Slices of the window range per head pair of the forward: one round of
// workgroups, two resident per CU.
static int win_fwd_pair_nslice(const Geo& g) {
  const int total = g.B * g.nwin;
  int target = 2 * g.cus / (g.heads / 2);
  if (target > total) target = total;
  if (target < 1) target = 1;
  return target;
}

template <bool QUAD, bool NHWC>
static void fwd_win_pair_go(const Geo& g, const void* q, const void* k, const void* v,
                            const float* table, void* o, float* lse, hipStream_t st) {
  const int total = g.B * g.nwin;
  const int nslice = win_fwd_pair_nslice(g);
  const int per = (total + nslice - 1) / nslice;
  const int grid = (g.heads / 2) * ((total + per - 1) / per);
  const float sl2 = kLog2e / sqrtf((float)g.hd);
  hipLaunchKernelGGL((fwd_win_pair_kernel<QUAD, NHWC>), dim3(grid), dim3(kPairThreads),
                     win_fwd_pair_lds(g), st, (const bf16*)q, (const bf16*)k, (const bf16*)v, table,
                     (bf16*)o, lse, g, per, sl2);
}

template <bool NHWC>
static void launch_win_fwd_t(const Geo& g, const void* q, const void* k, const void* v,
                             const float* table, void* o, float* lse, hipStream_t st) {
  const bool quad = quad_layout(g);
  if (g.hd == 32 && g.heads % 2 == 0) {
    if (quad) fwd_win_pair_go<true, NHWC>(g, q, k, v, table, o, lse, st);
    else fwd_win_pair_go<false, NHWC>(g, q, k, v, table, o, lse, st);
  } else if (g.hd == 32) {
    if (quad) fwd_win_go<32, true, NHWC>(g, q, k, v, table, o, lse, st);
    else fwd_win_go<32, false, NHWC>(g, q, k, v, table, o, lse, st);
  } else {
    if (quad) fwd_win_go<64, true, NHWC>(g, q, k, v, table, o, lse, st);
    else fwd_win_go<64, false, NHWC>(g, q, k, v, table, o, lse, st);
  }
}

hipError_t launch_win_fwd(const Geo& g, bool nhwc, const void* q, const void* k, const void* v,
                          const float* table, void* o, float* lse, hipStream_t st) {
  if (nhwc) launch_win_fwd_t<true>(g, q, k, v, table, o, lse, st);
  else launch_win_fwd_t<false>(g, q, k, v, table, o, lse, st);
  return hipGetLastError();
}

template <bool QUAD, bool NHWC>
static void bwd_win_go(const Geo& g, const void* q, const void* k, const void* v, const void* dout,
                       const float* lse, const float* table, void* dq, void* dk, void* dv,
                       float* partial, int nslice, hipStream_t st) {
  const int total = g.B * g.nwin;
  const int per = (total + nslice - 1) / nslice;
  const float sl2 = kLog2e / sqrtf((float)g.hd);
  const float scale = 1.0f / sqrtf((float)g.hd);
  hipLaunchKernelGGL((bwd_win_kernel<QUAD, NHWC>), dim3(g.heads * nslice), dim3(kWinThreads),
                     win_bwd_lds(g), st, (const bf16*)q, (const bf16*)k, (const bf16*)v,
                     (const bf16*)dout, lse, table, (bf16*)dq, (bf16*)dk, (bf16*)dv, partial, g,
                     nslice, per, sl2, scale);
}

hipError_t launch_win_bwd(const Geo& g, bool nhwc, const void* q, const void* k, const void* v,
                          const void* dout, const float* lse, const float* table, void* dq,
                          void* dk, void* dv, float* partial, int nslice, hipStream_t st) {
  const bool quad = quad_layout(g);
  if (nhwc) {
    if (quad) bwd_win_go<true, true>(g, q, k, v, dout, lse, table, dq, dk, dv, partial, nslice, st);
    else bwd_win_go<false, true>(g, q, k, v, dout, lse, table, dq, dk, dv, partial, nslice, st);
  } else {
    if (quad) bwd_win_go<true, false>(g, q, k, v, dout, lse, table, dq, dk, dv, partial, nslice, st);
    else bwd_win_go<false, false>(g, q, k, v, dout, lse, table, dq, dk, dv, partial, nslice, st);
  }
  return hipGetLastError();
}

}  // namespace terra
