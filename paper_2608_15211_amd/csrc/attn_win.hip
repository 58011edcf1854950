// attn_win.hip - window-resident attention kernels for windows of at most
// 128 tokens (bf16), the common Swin case (e.g. 8x8, 8x16 windows).
//
// Same mathematics as attn.hip (W-MSA / SW-MSA of the Swin blocks,
// Sec. IV-A, on the window-major layout of Sec. IV-D), organised so that a
// workgroup holds one whole window of one head:
// * every key of the window is in LDS at once, so the forward needs no
//   online rescaling and the backward has all of P and dP of a query in
//   registers: D_q = sum_k P dP is a register sum, and exp() runs once per
//   score in the backward;
// * 32x32 blocks are transposed ON THE MATRIX CORES: multiplying a block by
//   a 0/1 permutation operand returns it in the transposed register layout
//   (values are exact bf16, so the copy is exact).  This gives K^T and V^T
//   for LDS, the query-major Q and dO operands, and P^T, dS^T for dK/dV
//   without recomputing the scores;
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
  const int a = t / cols;
  const int c = t - a * cols;
  const int lab = row_label(g, i * g.wh + a) | col_label(g, j * g.ww + c);
  return (a * g.bstride + c) | (lab << 24);
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
template <int HD>
__device__ inline void stage_rows(const bf16* __restrict__ src, int64_t tok0, int n, int C,
                                  int hoff, bf16* lds) {
  constexpr int kCpr = HD / 8;
  for (int idx = threadIdx.x; idx < kWinMax * kCpr; idx += kWinThreads) {
    const int row = idx / kCpr;
    const int ch = idx - row * kCpr;
    uint4 raw = make_uint4(0, 0, 0, 0);
    if (row < n) raw = *reinterpret_cast<const uint4*>(src + (tok0 + row) * C + hoff + ch * 8);
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
  const bool lat = (g.flags & 1) && g.sh > 0 && (wi * g.wh + win_rows(g, wi)) > g.H - g.sh;
  const bool lon = (g.flags & 2) && g.sw > 0 && (wj * g.ww + win_cols(g, wj)) > g.W - g.sw;
  return lat || lon || (n & 31) != 0;
}

// Accumulator initialiser of key block KB: the bias of each (query, key)
// pair, pre-multiplied by sqrt(hd) so that one multiply by log2(e)/sqrt(hd)
// after the QK^T product yields the log2-domain score; -inf for excluded
// pairs (tab[nbins .. nbins+3] holds -inf).  qrev is the lane's reversed
// bin offset, qlab its label.
template <bool QUAD, bool MASK>
__device__ inline f32x16 bias_init(const int* kinfo, const float* tab, int kb, int half, int qrev,
                                   int qlab, int nbins) {
  f32x16 c;
#pragma unroll
  for (int g4 = 0; g4 < 4; ++g4) {
    int inf = kinfo[32 * kb + 8 * g4 + 4 * half];
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      if (!QUAD && x > 0) inf = kinfo[32 * kb + 8 * g4 + 4 * half + x];
      int rb = qrev + (inf & 0xFFFFFF);
      if (MASK && (inf >> 24) != qlab) rb = nbins - (QUAD ? x : 0);
      c[4 * g4 + x] = tab[rb + (QUAD ? x : 0)];
    }
  }
  return c;
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
template <int HD, bool QUAD>
__global__ __launch_bounds__(kWinThreads) void fwd_win_kernel(
    const bf16* __restrict__ q, const bf16* __restrict__ k, const bf16* __restrict__ v,
    const float* __restrict__ table, bf16* __restrict__ o, float* __restrict__ lse, Geo g,
    float scale_log2) {
  extern __shared__ __align__(16) char smem[];
  bf16* ks = reinterpret_cast<bf16*>(smem);                       // [128][HD+8]
  bf16* vts = ks + kWinMax * (HD + 8);                            // [HD][128+8]
  int* kinfo = reinterpret_cast<int*>(vts + HD * (kWinMax + 8));  // [128]
  float* tab = reinterpret_cast<float*>(kinfo + kWinMax);         // [nbins]

  int work = xcd_work(blockIdx.x, gridDim.x);
  const int h = work % g.heads; work /= g.heads;
  const int w = work % g.nwin;
  const int b = work / g.nwin;
  const int wi = w / g.Mw, wj = w - (w / g.Mw) * g.Mw;
  const int cols = win_cols(g, wj);
  const int n = win_rows(g, wi) * cols;
  const int nkb = (n + 31) >> 5;
  const int64_t img0 = (int64_t)b * g.HW;
  const int64_t tok0 = img0 + win_offset(g, wi, wj);
  const int hoff = h * HD;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, col = lane & 31;

  // bias table of head h times sqrt(hd), stored in reverse bin order so that
  // consecutive keys of a window row read consecutive addresses; four -inf
  // entries after it serve excluded pairs
  const float bscale = sqrtf((float)HD);
  for (int x = threadIdx.x; x < g.nbins + 4; x += kWinThreads)
    tab[x] = x < g.nbins ? table[(g.nbins - 1 - x) * g.heads + h] * bscale : -INFINITY;
  if (threadIdx.x < kWinMax) kinfo[threadIdx.x] = win_token_info(g, wi, wj, cols, threadIdx.x, n);
  stage_rows<HD>(k, tok0, n, g.C, hoff, ks);
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
        const bf16* p = v + (tok0 + row) * g.C + hoff + 32 * eb + 8 * half;
        a0 = *reinterpret_cast<const bf16x8*>(p);
        a1 = *reinterpret_cast<const bf16x8*>(p + 16);
      }
      const f32x16 t = mfma_transpose(a0, a1, i0, i1);
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4)
        store4_bf16(vts + (32 * eb + col) * (kWinMax + 8) + 32 * wave + 8 * g4 + 4 * half, t, g4, 1.0f);
    }
  }
  __syncthreads();
  if (wave >= nkb) return;

  const int qi = 32 * wave + col;
  const bool qvalid = qi < n;
  const int qinf = kinfo[qvalid ? qi : 0];
  const int qlab = qinf >> 24;
  // reversed bin of (q, k) = qrev + koff(k)
  const int qrev = g.nbins - 1 - ((qinf & 0xFFFFFF) + (g.wh - 1) * g.bstride + (g.ww - 1));
  bf16x8 qop[HD / 16];
#pragma unroll
  for (int c = 0; c < HD / 16; ++c)
    qop[c] = qvalid ? *reinterpret_cast<const bf16x8*>(q + (tok0 + qi) * g.C + hoff + 16 * c + 8 * half)
                    : zero8();

  // raw scores with the bias folded into the accumulator: s = QK^T + bias*sqrt(hd)
  f32x16 s[4];
  const bool mask = window_needs_mask(g, wi, wj, n);
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    if (kb < nkb) {
      s[kb] = mask ? bias_init<QUAD, true>(kinfo, tab, kb, half, qrev, qlab, g.nbins)
                   : bias_init<QUAD, false>(kinfo, tab, kb, half, qrev, qlab, g.nbins);
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
  mr = fmaxf(mr, __shfl_xor(mr, 32));
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
  l += __shfl_xor(l, 32);
  if (!qvalid) return;
  const float inv = 1.0f / l;
  bf16* orow = o + (tok0 + qi) * g.C + hoff;
#pragma unroll
  for (int eb = 0; eb < HD / 32; ++eb)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) store4_bf16(orow + 32 * eb + 8 * g4 + 4 * half, oacc[eb], g4, inv);
  if (half == 0) lse[(img0 * g.heads) + (int64_t)h * g.HW + (tok0 - img0) + qi] = (m + __log2f(l)) * kLn2;
}

// ---------------------------------------------------------------------------
// Forward for head_dim 32 and an even head count: one workgroup of 8 waves
// per (image, window, head pair).  Global memory is touched only in
// row-contiguous 128-byte segments (8 lanes per token row): Q, K and V are
// staged through LDS (V transposed by the staging stores) and O goes back
// through LDS.  Wave w handles head 2*hp + (w >> 2) and queries
// [32*(w&3), 32*(w&3)+32).
// ---------------------------------------------------------------------------
constexpr int kPairThreads = 512;

template <bool QUAD>
__global__ __launch_bounds__(kPairThreads) void fwd_win_pair_kernel(
    const bf16* __restrict__ q, const bf16* __restrict__ k, const bf16* __restrict__ v,
    const float* __restrict__ table, bf16* __restrict__ o, float* __restrict__ lse, Geo g,
    float scale_log2) {
  constexpr int HD = 32;
  constexpr int KS = HD + 8, VS = kWinMax + 8;
  extern __shared__ __align__(16) char smem[];
  bf16* ks = reinterpret_cast<bf16*>(smem);                        // [2][128][KS] K rows
  bf16* qs = ks + 2 * kWinMax * KS;                                // [2][128][KS] Q rows, then O
  bf16* vts = qs + 2 * kWinMax * KS;                               // [2][HD][VS]  V^T
  int* kinfo = reinterpret_cast<int*>(vts + 2 * HD * VS);          // [128]
  float* tab = reinterpret_cast<float*>(kinfo + kWinMax);          // [2][nbins+4]

  const int hpairs = g.heads >> 1;
  int work = xcd_work(blockIdx.x, gridDim.x);
  const int hp = work % hpairs; work /= hpairs;
  const int w = work % g.nwin;
  const int b = work / g.nwin;
  const int wi = w / g.Mw, wj = w - (w / g.Mw) * g.Mw;
  const int cols = win_cols(g, wj);
  const int n = win_rows(g, wi) * cols;
  const int nkb = (n + 31) >> 5;
  const int64_t img0 = (int64_t)b * g.HW;
  const int64_t tok0 = img0 + win_offset(g, wi, wj);
  const int64_t cbase = (int64_t)2 * hp * HD;          // first channel of the pair
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int hs = wave >> 2, qb = wave & 3;
  const int h = 2 * hp + hs;
  const int qi = 32 * qb + col;
  const bool qvalid = qi < n;

  // ---- row-contiguous loads: thread -> (row, 16-byte chunk of the pair) ----
  uint4 kr[2], qr[2], vr[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int idx = threadIdx.x + u * kPairThreads;
    const int row = idx >> 3, ch = idx & 7;
    kr[u] = qr[u] = vr[u] = make_uint4(0, 0, 0, 0);
    if (row < n) {
      const int64_t off = (tok0 + row) * g.C + cbase + ch * 8;
      kr[u] = *reinterpret_cast<const uint4*>(k + off);
      qr[u] = *reinterpret_cast<const uint4*>(q + off);
      vr[u] = *reinterpret_cast<const uint4*>(v + off);
    }
  }
  const float bscale = sqrtf((float)HD);
  for (int x = threadIdx.x; x < 2 * (g.nbins + 4); x += kPairThreads) {
    const int t = x / (g.nbins + 4), y = x - t * (g.nbins + 4);
    tab[x] = y < g.nbins ? table[(g.nbins - 1 - y) * g.heads + 2 * hp + t] * bscale : -INFINITY;
  }
  if (threadIdx.x < kWinMax) kinfo[threadIdx.x] = win_token_info(g, wi, wj, cols, threadIdx.x, n);
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int idx = threadIdx.x + u * kPairThreads;
    const int row = idx >> 3, ch = idx & 7;
    const int t = ch >> 2, e0 = (ch & 3) * 8;
    *reinterpret_cast<uint4*>(ks + (t * kWinMax + row) * KS + e0) = kr[u];
    *reinterpret_cast<uint4*>(qs + (t * kWinMax + row) * KS + e0) = qr[u];
    const bf16* ve = reinterpret_cast<const bf16*>(&vr[u]);
#pragma unroll
    for (int x = 0; x < 8; ++x) vts[(t * HD + e0 + x) * VS + row] = ve[x];
  }
  __syncthreads();

  const bool active = qb < nkb;
  const bf16* ksh = ks + hs * kWinMax * KS;
  const bf16* vth = vts + hs * HD * VS;
  const float* tabh = tab + hs * (g.nbins + 4);
  f32x16 oacc = f32x16{};
  float m = 0.0f, l = 1.0f;
  if (active) {
    bf16x8 qop[2];
#pragma unroll
    for (int c = 0; c < 2; ++c)
      qop[c] = *reinterpret_cast<const bf16x8*>(qs + (hs * kWinMax + qi) * KS + 16 * c + 8 * half);
    const int qinf = kinfo[qvalid ? qi : 0];
    const int qlab = qinf >> 24;
    const int qrev = g.nbins - 1 - ((qinf & 0xFFFFFF) + (g.wh - 1) * g.bstride + (g.ww - 1));
    const bool mask = window_needs_mask(g, wi, wj, n);
    f32x16 s[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      if (kb < nkb) {
        s[kb] = mask ? bias_init<QUAD, true>(kinfo, tabh, kb, half, qrev, qlab, g.nbins)
                     : bias_init<QUAD, false>(kinfo, tabh, kb, half, qrev, qlab, g.nbins);
#pragma unroll
        for (int c = 0; c < 2; ++c)
          mma16(s[kb], *reinterpret_cast<const bf16x8*>(ksh + (32 * kb + col) * KS + 16 * c + 8 * half), qop[c]);
      }
    }
    float mr = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
      if (kb < nkb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mr = fmaxf(mr, s[kb][r]);
    mr = fmaxf(mr, __shfl_xor(mr, 32));
    m = mr * scale_log2;
    l = 0.0f;
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
        for (int c = 0; c < 2; ++c)
          mma16(oacc, lds_perm_op(vth + col * VS + 32 * kb + 16 * c, half), pack_bf16(s[kb], 8 * c));
      }
    }
    l += __shfl_xor(l, 32);
  }
  __syncthreads();   // every wave has read its Q rows; qs now takes O
  if (active) {
    const float inv = 1.0f / l;
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4)
      store4_bf16(qs + (hs * kWinMax + qi) * KS + 8 * g4 + 4 * half, oacc, g4, inv);
    if (qvalid && half == 0)
      lse[(img0 * g.heads) + (int64_t)h * g.HW + (tok0 - img0) + qi] = (m + __log2f(l)) * kLn2;
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int idx = threadIdx.x + u * kPairThreads;
    const int row = idx >> 3, ch = idx & 7;
    if (row < n) {
      const int t = ch >> 2, e0 = (ch & 3) * 8;
      *reinterpret_cast<uint4*>(o + (tok0 + row) * g.C + cbase + ch * 8) =
          *reinterpret_cast<const uint4*>(qs + (t * kWinMax + row) * KS + e0);
    }
  }
}

// ---------------------------------------------------------------------------
// Backward (head_dim 32): one workgroup per (head, run of windows).  Per
// window: wave w owns queries [32w, 32w+32) for P, dP, D, dS and dQ, then
// the four waves rotate over the key blocks to sum dV and dK in LDS.
// ---------------------------------------------------------------------------
constexpr int kBwdHD = 32;

// Identity operands kept in LDS (re-read at each use so that they do not
// occupy registers across the window loop): [natural c0, c1, permuted c0, c1][lane].
__device__ inline bf16x8 lds_ident(const bf16x8* id, int which) {
  return id[which * 64 + (threadIdx.x & 63)];
}

// Everything one wave needs for the per-key-block steps of one window.
struct BwdStep {
  const bf16* vs;       // V rows in LDS
  const bf16* kts;      // K^T in LDS
  const bf16x8* ident;
  float* redv;          // dV partial sums [HD][RS]
  float* redk;          // dK partial sums [HD][RS]
  bf16x8 dop[2];        // dO of the wave's queries (row operand)
  bf16x8 de[2], qe[2];  // dO and Q with lane = channel (column operand)
  float D;
  int col, half;
};

// Key block KB of the wave: dP (recomputed), dS, the bias accumulators,
// the dQ contribution, and the dV / dK partials added into LDS.  T is the
// rotation step (0 stores, later steps add).
template <int KB, int T>
__device__ inline void bwd_key_block(const BwdStep& st, const f32x16& p, f32x16& dtacc,
                                     f32x16& dqacc) {
  constexpr int HD = kBwdHD;
  constexpr int RS = kWinMax + 4;
  f32x16 ds = f32x16{};
#pragma unroll
  for (int c = 0; c < 2; ++c)
    mma16(ds, *reinterpret_cast<const bf16x8*>(st.vs + (32 * KB + st.col) * (HD + 8) + 16 * c + 8 * st.half),
          st.dop[c]);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    ds[r] = p[r] * (ds[r] - st.D);
    dtacc[r] += ds[r];
  }
  const bf16x8 pb0 = pack_bf16(p, 0), pb1 = pack_bf16(p, 8);
  const bf16x8 db0 = pack_bf16(ds, 0), db1 = pack_bf16(ds, 8);
  mma16(dqacc, lds_perm_op(st.kts + st.col * (kWinMax + 8) + 32 * KB, st.half), db0);
  mma16(dqacc, lds_perm_op(st.kts + st.col * (kWinMax + 8) + 32 * KB + 16, st.half), db1);
  // (P or dS)^T of this block has lane = key; times dO or Q (lane = channel)
  const f32x16 tp = mfma_transpose(pb0, pb1, lds_ident(st.ident, 2), lds_ident(st.ident, 3));
  const f32x16 td = mfma_transpose(db0, db1, lds_ident(st.ident, 2), lds_ident(st.ident, 3));
  // partials: lane = channel, registers = keys 32KB + acc_row(r, half); the
  // running sums from earlier steps enter as the accumulator input
  f32x16 pv, pk;
#pragma unroll
  for (int g4 = 0; g4 < 4; ++g4) {
    const int off = st.col * RS + 32 * KB + 8 * g4 + 4 * st.half;
    const f32x4 a = T > 0 ? *reinterpret_cast<const f32x4*>(st.redv + off) : f32x4{0.f, 0.f, 0.f, 0.f};
    const f32x4 b = T > 0 ? *reinterpret_cast<const f32x4*>(st.redk + off) : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int x = 0; x < 4; ++x) { pv[4 * g4 + x] = a[x]; pk[4 * g4 + x] = b[x]; }
  }
  mma16(pv, pack_bf16(tp, 0), st.de[0]);
  mma16(pv, pack_bf16(tp, 8), st.de[1]);
  mma16(pk, pack_bf16(td, 0), st.qe[0]);
  mma16(pk, pack_bf16(td, 8), st.qe[1]);
#pragma unroll
  for (int g4 = 0; g4 < 4; ++g4) {
    const int off = st.col * RS + 32 * KB + 8 * g4 + 4 * st.half;
    *reinterpret_cast<f32x4*>(st.redv + off) = f32x4{pv[4 * g4], pv[4 * g4 + 1], pv[4 * g4 + 2], pv[4 * g4 + 3]};
    *reinterpret_cast<f32x4*>(st.redk + off) = f32x4{pk[4 * g4], pk[4 * g4 + 1], pk[4 * g4 + 2], pk[4 * g4 + 3]};
  }
}

// The four steps of wave W: key blocks W, W+1, W+2, W+3 (mod 4), so that at
// every step each block is touched by exactly one wave; a barrier ends each
// step.  The order of additions into every block is therefore fixed.
template <int W>
__device__ inline void bwd_rotation(const BwdStep& st, const f32x16 (&p)[4], f32x16 (&dtacc)[4],
                                    f32x16& dqacc) {
  bwd_key_block<(W + 0) & 3, 0>(st, p[(W + 0) & 3], dtacc[(W + 0) & 3], dqacc);
  __syncthreads();
  bwd_key_block<(W + 1) & 3, 1>(st, p[(W + 1) & 3], dtacc[(W + 1) & 3], dqacc);
  __syncthreads();
  bwd_key_block<(W + 2) & 3, 2>(st, p[(W + 2) & 3], dtacc[(W + 2) & 3], dqacc);
  __syncthreads();
  bwd_key_block<(W + 3) & 3, 3>(st, p[(W + 3) & 3], dtacc[(W + 3) & 3], dqacc);
  __syncthreads();
}

template <bool QUAD>
__global__ __launch_bounds__(kWinThreads) void bwd_win_kernel(
    const bf16* __restrict__ q, const bf16* __restrict__ k, const bf16* __restrict__ v,
    const bf16* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ table,
    bf16* __restrict__ dq, bf16* __restrict__ dk, bf16* __restrict__ dv,
    float* __restrict__ partial, Geo g, int nslice, int per_slice, float scale_log2, float scale) {
  constexpr int HD = kBwdHD;
  constexpr int RS = kWinMax + 4;                               // red row stride (floats)
  extern __shared__ __align__(16) char smem[];
  bf16x8* ident = reinterpret_cast<bf16x8*>(smem);              // [4][64]
  bf16* ks = reinterpret_cast<bf16*>(ident + 4 * 64);           // K   [128][HD+8]
  bf16* vs = ks + kWinMax * (HD + 8);                           // V   [128][HD+8]
  bf16* kts = vs + kWinMax * (HD + 8);                          // K^T [HD][128+8]
  float* redv = reinterpret_cast<float*>(kts + HD * (kWinMax + 8));  // [HD][RS]
  float* redk = redv + HD * RS;                                 // [HD][RS]
  int* kinfo = reinterpret_cast<int*>(redk + HD * RS);          // [128]
  float* tab = reinterpret_cast<float*>(kinfo + kWinMax);       // [nbins], reversed
  float* dtb = tab + g.nbins + 4;                               // [4][nbins], reversed

  const int work = xcd_work(blockIdx.x, gridDim.x);
  const int slice = work / g.heads;
  const int h = work - slice * g.heads;
  const int hoff = h * HD;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int half = lane >> 5, col = lane & 31;
  float* mybins = dtb + wave * g.nbins;

  for (int x = threadIdx.x; x < g.nbins; x += kWinThreads) {
#pragma unroll
    for (int w4 = 0; w4 < 4; ++w4) dtb[w4 * g.nbins + x] = 0.0f;
  }
  // bias table times sqrt(hd), reversed bin order, then four -inf entries
  for (int x = threadIdx.x; x < g.nbins + 4; x += kWinThreads)
    tab[x] = x < g.nbins ? table[(g.nbins - 1 - x) * g.heads + h] * sqrtf((float)HD) : -INFINITY;
  if (wave == 0) {
    ident[0 * 64 + lane] = ident_op<false>(0);
    ident[1 * 64 + lane] = ident_op<false>(1);
    ident[2 * 64 + lane] = ident_op<true>(0);
    ident[3 * 64 + lane] = ident_op<true>(1);
  }

  // Bias-gradient accumulators, one per result register.  A register holds
  // the same (query slot, key slot) pair in every window, and the pair's
  // bin depends only on the window width, so dS is summed here over a run
  // of windows of equal width and flushed to the per-wave LDS bins (in the
  // same fixed order every time) when the width changes.
  f32x16 dtacc[4];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) dtacc[kb] = f32x16{};
  int acc_cols = 0;
  // (hh is made opaque so that the per-register key slots below are not
  // hoisted out of the window loop into 64 live registers)
#define TERRA_FLUSH_DT(cw)                                                              \
  {                                                                                     \
    const float rcw = 1.0f / (float)(cw);                                               \
    const int qs = 32 * wave + col;                                                     \
    const int aq = (int)(((float)qs + 0.5f) * rcw), cq = qs - aq * (cw);                \
    int hh = half;                                                                      \
    asm volatile("" : "+v"(hh));                                                        \
    _Pragma("unroll") for (int kb = 0; kb < 4; ++kb)                                    \
    _Pragma("unroll") for (int r = 0; r < 16; ++r) {                                    \
      const int kk = 32 * kb + acc_row(r, hh);                                          \
      const int ak = (int)(((float)kk + 0.5f) * rcw), ck = kk - ak * (cw);              \
      if (aq < g.wh && ak < g.wh)                                                       \
        atomicAdd(&mybins[g.nbins - 1 - ((aq - ak + g.wh - 1) * g.bstride +             \
                                         (cq - ck + g.ww - 1))], dtacc[kb][r]);         \
      dtacc[kb][r] = 0.0f;                                                              \
    }                                                                                   \
  }

  const int total = g.B * g.nwin;
  const int wbeg = slice * per_slice;
  const int wend = min(total, wbeg + per_slice);

  // Global loads of the next window are issued before the current window is
  // computed, so their latency overlaps the work: K and V rows for LDS
  // staging (2 x 16 B of each per thread), Q and dO of the lane's query and
  // its log-sum-exp.
  uint4 kpre[2], vpre[2];
  bf16x8 qpre[2], dpre[2];
  float lpre = 0.0f;
  auto prefetch = [&](int wl) {
    const int b = wl / g.nwin;
    const int w = wl - b * g.nwin;
    const int wi = w / g.Mw, wj = w - (w / g.Mw) * g.Mw;
    const int n = win_rows(g, wi) * win_cols(g, wj);
    const int64_t img0 = (int64_t)b * g.HW;
    const int64_t tok0 = img0 + win_offset(g, wi, wj);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int idx = threadIdx.x + u * kWinThreads;
      const int row = idx >> 2, ch = idx & 3;
      kpre[u] = make_uint4(0, 0, 0, 0);
      vpre[u] = make_uint4(0, 0, 0, 0);
      if (row < n) {
        kpre[u] = *reinterpret_cast<const uint4*>(k + (tok0 + row) * g.C + hoff + ch * 8);
        vpre[u] = *reinterpret_cast<const uint4*>(v + (tok0 + row) * g.C + hoff + ch * 8);
      }
    }
    const int qi = 32 * wave + col;
    const bool qvalid = qi < n;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      qpre[c] = qvalid ? *reinterpret_cast<const bf16x8*>(q + (tok0 + qi) * g.C + hoff + 16 * c + 8 * half)
                       : zero8();
      dpre[c] = qvalid ? *reinterpret_cast<const bf16x8*>(dout + (tok0 + qi) * g.C + hoff + 16 * c + 8 * half)
                       : zero8();
    }
    // (+inf for padding queries makes every P of theirs exactly 0)
    lpre = qvalid ? lse[img0 * g.heads + (int64_t)h * g.HW + (tok0 - img0) + qi] * kLog2e : INFINITY;
  };
  if (wbeg < wend) prefetch(wbeg);

  for (int wl = wbeg; wl < wend; ++wl) {
    const int b = wl / g.nwin;
    const int w = wl - b * g.nwin;
    const int wi = w / g.Mw, wj = w - (w / g.Mw) * g.Mw;
    const int cols = win_cols(g, wj);
    const int n = win_rows(g, wi) * cols;
    const int64_t img0 = (int64_t)b * g.HW;
    const int64_t tok0 = img0 + win_offset(g, wi, wj);
    if (cols != acc_cols) {          // uniform across the workgroup
      if (acc_cols > 0) TERRA_FLUSH_DT(acc_cols);
      acc_cols = cols;
    }

    __syncthreads();   // the previous window is done with LDS
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int idx = threadIdx.x + u * kWinThreads;
      const int row = idx >> 2, ch = idx & 3;
      *reinterpret_cast<uint4*>(ks + row * (HD + 8) + ch * 8) = kpre[u];
      *reinterpret_cast<uint4*>(vs + row * (HD + 8) + ch * 8) = vpre[u];
    }
    if (threadIdx.x < kWinMax) kinfo[threadIdx.x] = win_token_info(g, wi, wj, cols, threadIdx.x, n);
    BwdStep st;
    bf16x8 qop[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      qop[c] = qpre[c];
      st.dop[c] = dpre[c];
    }
    const float lse2 = lpre;
    if (wl + 1 < wend) prefetch(wl + 1);
    __syncthreads();
    {
      // K^T: wave w transposes keys [32w, 32w+32) on the matrix cores
      const bf16* r = ks + (32 * wave + col) * (HD + 8) + 8 * half;
      const f32x16 t = mfma_transpose(*reinterpret_cast<const bf16x8*>(r),
                                      *reinterpret_cast<const bf16x8*>(r + 16),
                                      lds_ident(ident, 0), lds_ident(ident, 1));
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4)
        store4_bf16(kts + col * (kWinMax + 8) + 32 * wave + 8 * g4 + 4 * half, t, g4, 1.0f);
    }

    // ---- the wave's 32 queries (32*wave + col) ----
    const int qi = 32 * wave + col;
    const bool qvalid = qi < n;
    const int qinf = qvalid ? win_token_info(g, wi, wj, cols, qi, n) : 0;
    const int qlab = qinf >> 24;
    const int qrev = g.nbins - 1 - ((qinf & 0xFFFFFF) + (g.wh - 1) * g.bstride + (g.ww - 1));

    // scores (transposed: lane = query, registers = keys) with the bias in
    // the accumulator, P, and D = sum P dP
    const bool mask = window_needs_mask(g, wi, wj, n);
    f32x16 p[4];
    float dsum = 0.0f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      f32x16 dp = f32x16{};
      p[kb] = mask ? bias_init<QUAD, true>(kinfo, tab, kb, half, qrev, qlab, g.nbins)
                   : bias_init<QUAD, false>(kinfo, tab, kb, half, qrev, qlab, g.nbins);
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        mma16(p[kb], *reinterpret_cast<const bf16x8*>(ks + (32 * kb + col) * (HD + 8) + 16 * c + 8 * half), qop[c]);
        mma16(dp, *reinterpret_cast<const bf16x8*>(vs + (32 * kb + col) * (HD + 8) + 16 * c + 8 * half), st.dop[c]);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float pv = __builtin_amdgcn_exp2f(p[kb][r] * scale_log2 - lse2);
        p[kb][r] = pv;
        dsum += pv * dp[r];
      }
    }
    st.D = dsum + __shfl_xor(dsum, 32);
    // dP is recomputed per key block on the matrix cores rather than kept in
    // 64 registers (the fence stops the compiler from reusing the first one).
    asm volatile("" ::: "memory");
    {
      const f32x16 te = mfma_transpose(st.dop[0], st.dop[1], lds_ident(ident, 0), lds_ident(ident, 1));
      st.de[0] = pack_bf16(te, 0);
      st.de[1] = pack_bf16(te, 8);
      const f32x16 tq = mfma_transpose(qop[0], qop[1], lds_ident(ident, 0), lds_ident(ident, 1));
      st.qe[0] = pack_bf16(tq, 0);
      st.qe[1] = pack_bf16(tq, 8);
    }
    st.vs = vs;
    st.kts = kts;
    st.ident = ident;
    st.redv = redv;
    st.redk = redk;
    st.col = col;
    st.half = half;
    __syncthreads();   // K^T complete
    f32x16 dqacc = f32x16{};
    switch (wave) {
      case 0: bwd_rotation<0>(st, p, dtacc, dqacc); break;
      case 1: bwd_rotation<1>(st, p, dtacc, dqacc); break;
      case 2: bwd_rotation<2>(st, p, dtacc, dqacc); break;
      default: bwd_rotation<3>(st, p, dtacc, dqacc); break;
    }
    if (qvalid) {
      bf16* row = dq + (tok0 + qi) * g.C + hoff;
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) store4_bf16(row + 8 * g4 + 4 * half, dqacc, g4, scale);
    }
    // dV and dK of the window: thread -> (key, 16 channels)
    {
      const int key = threadIdx.x >> 1;
      const int c0 = (threadIdx.x & 1) * 16;
      if (key < n) {
        bf16x8 lo, hi;
#pragma unroll
        for (int x = 0; x < 8; ++x) {
          lo[x] = (bf16)redv[(c0 + x) * RS + key];
          hi[x] = (bf16)redv[(c0 + 8 + x) * RS + key];
        }
        bf16* dst = dv + (tok0 + key) * g.C + hoff + c0;
        *reinterpret_cast<bf16x8*>(dst) = lo;
        *reinterpret_cast<bf16x8*>(dst + 8) = hi;
#pragma unroll
        for (int x = 0; x < 8; ++x) {
          lo[x] = (bf16)(redk[(c0 + x) * RS + key] * scale);
          hi[x] = (bf16)(redk[(c0 + 8 + x) * RS + key] * scale);
        }
        dst = dk + (tok0 + key) * g.C + hoff + c0;
        *reinterpret_cast<bf16x8*>(dst) = lo;
        *reinterpret_cast<bf16x8*>(dst + 8) = hi;
      }
    }
  }
  if (acc_cols > 0) TERRA_FLUSH_DT(acc_cols);
#undef TERRA_FLUSH_DT
  __syncthreads();
  float* out = partial + ((int64_t)h * nslice + slice) * g.nbins;
  for (int x = threadIdx.x; x < g.nbins; x += kWinThreads) {
    const int rx = g.nbins - 1 - x;
    out[x] = ((dtb[rx] + dtb[g.nbins + rx]) + dtb[2 * g.nbins + rx]) + dtb[3 * g.nbins + rx];
  }
}

// ---------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------
bool win_fwd_ok(const Geo& g, bool bf16_) { return bf16_ && g.wh * g.ww <= kWinMax && (g.hd == 32 || g.hd == 64); }
bool win_bwd_ok(const Geo& g, bool bf16_) { return bf16_ && g.wh * g.ww <= kWinMax && g.hd == kBwdHD; }

// Slices of the window range per head; a pure function of the geometry.
int win_bwd_nslice(const Geo& g) {
  const int total = g.B * g.nwin;
  int target = (1024 + g.heads - 1) / g.heads;     // ~1024 workgroups
  if (target > total) target = total;
  if (target < 1) target = 1;
  const int per = (total + target - 1) / target;
  return (total + per - 1) / per;
}

size_t win_fwd_pair_lds(const Geo& g);
size_t win_fwd_lds(const Geo& g) {
  const size_t one = sizeof(bf16) * (kWinMax * (g.hd + 8) + g.hd * (kWinMax + 8)) + 4 * kWinMax +
                     4 * (g.nbins + 4);
  if (g.hd == 32 && g.heads % 2 == 0) {
    const size_t pair = win_fwd_pair_lds(g);
    return pair > one ? pair : one;
  }
  return one;
}
size_t win_bwd_lds(const Geo& g) {
  return 4 * 64 * sizeof(bf16x8) + sizeof(bf16) * (2 * kWinMax * (kBwdHD + 8) + kBwdHD * (kWinMax + 8)) +
         2 * 4 * kBwdHD * (kWinMax + 4) + 4 * kWinMax + 4 * (5 * g.nbins + 4);
}

// Four consecutive result registers are four consecutive keys of one window
// row, with one label, when every window width is a multiple of 4 and the
// longitude wrap is not masked.
static bool quad_layout(const Geo& g) {
  return g.ww % 4 == 0 && (g.W % g.ww) % 4 == 0 && (g.flags & 2) == 0;
}

template <int HD, bool QUAD>
static void fwd_win_go(const Geo& g, const void* q, const void* k, const void* v,
                       const float* table, void* o, float* lse, hipStream_t st) {
  const int grid = g.B * g.nwin * g.heads;
  const float sl2 = kLog2e / sqrtf((float)g.hd);
  hipLaunchKernelGGL((fwd_win_kernel<HD, QUAD>), dim3(grid), dim3(kWinThreads), win_fwd_lds(g), st,
                     (const bf16*)q, (const bf16*)k, (const bf16*)v, table, (bf16*)o, lse, g, sl2);
}

size_t win_fwd_pair_lds(const Geo& g) {
  return sizeof(bf16) * 2 * (2 * kWinMax * (32 + 8) + 32 * (kWinMax + 8)) + 4 * kWinMax +
         4 * 2 * (g.nbins + 4);
}

hipError_t launch_win_fwd(const Geo& g, const void* q, const void* k, const void* v,
                          const float* table, void* o, float* lse, hipStream_t st) {
  const bool quad = quad_layout(g);
  if (g.hd == 32 && g.heads % 2 == 0) {
    const int grid = g.B * g.nwin * (g.heads / 2);
    const float sl2 = kLog2e / sqrtf((float)g.hd);
    if (quad)
      hipLaunchKernelGGL((fwd_win_pair_kernel<true>), dim3(grid), dim3(kPairThreads),
                         win_fwd_pair_lds(g), st, (const bf16*)q, (const bf16*)k, (const bf16*)v,
                         table, (bf16*)o, lse, g, sl2);
    else
      hipLaunchKernelGGL((fwd_win_pair_kernel<false>), dim3(grid), dim3(kPairThreads),
                         win_fwd_pair_lds(g), st, (const bf16*)q, (const bf16*)k, (const bf16*)v,
                         table, (bf16*)o, lse, g, sl2);
    return hipGetLastError();
  }
  if (g.hd == 32) {
    if (quad) fwd_win_go<32, true>(g, q, k, v, table, o, lse, st);
    else fwd_win_go<32, false>(g, q, k, v, table, o, lse, st);
  } else {
    if (quad) fwd_win_go<64, true>(g, q, k, v, table, o, lse, st);
    else fwd_win_go<64, false>(g, q, k, v, table, o, lse, st);
  }
  return hipGetLastError();
}

hipError_t launch_win_bwd(const Geo& g, const void* q, const void* k, const void* v,
                          const void* dout, const float* lse, const float* table, void* dq,
                          void* dk, void* dv, float* partial, int nslice, hipStream_t st) {
  const int total = g.B * g.nwin;
  const int per = (total + nslice - 1) / nslice;
  const float sl2 = kLog2e / sqrtf((float)g.hd);
  const float scale = 1.0f / sqrtf((float)g.hd);
  if (quad_layout(g))
    hipLaunchKernelGGL((bwd_win_kernel<true>), dim3(g.heads * nslice), dim3(kWinThreads),
                       win_bwd_lds(g), st, (const bf16*)q, (const bf16*)k, (const bf16*)v,
                       (const bf16*)dout, lse, table, (bf16*)dq, (bf16*)dk, (bf16*)dv, partial, g,
                       nslice, per, sl2, scale);
  else
    hipLaunchKernelGGL((bwd_win_kernel<false>), dim3(g.heads * nslice), dim3(kWinThreads),
                       win_bwd_lds(g), st, (const bf16*)q, (const bf16*)k, (const bf16*)v,
                       (const bf16*)dout, lse, table, (bf16*)dq, (bf16*)dk, (bf16*)dv, partial, g,
                       nslice, per, sl2, scale);
  return hipGetLastError();
}

}  // namespace terra
