// attn.hip - shifted-window multi-head self-attention for gfx950.
//
// The Swin blocks of the paper (Sec. IV-A, W-MSA / SW-MSA) attend inside
// each window of the window-major layout built by the token route
// (Sec. IV-D).  Per window and head:
//   S = Q K^T / sqrt(hd) + T[bin(q, k)],  masked pairs excluded,
//   P = softmax(S),  O = P V,  LSE = ln sum_k exp S
// and the backward
//   dV = P^T dO,  dP = dO V^T,  dS = P (dP - D),  D_q = sum_k P dP,
//   dQ = dS K / sqrt(hd),  dK = dS^T Q / sqrt(hd),  dT[bin] = sum dS.
//
// Kernel design (CDNA4, wave64):
// * QK^T, PV, dO V^T, dS K, dS^T Q and P^T dO run on the matrix cores
//   (32x32x16 bf16, or 32x32x2 fp32 for the fp32 path), fp32 accumulate.
// * A wave owns 32 queries (forward, dQ) or 32 keys (dK/dV).  The score
//   tile is produced TRANSPOSED where its rows must feed the next product
//   from registers: the result layout of one MFMA is then directly the
//   register operand of the next, with the contraction order permuted
//   consistently on the LDS side (no register shuffles).
// * K/V (forward, dQ) or Q/dO (dK/dV) tiles of 64 tokens are staged in LDS
//   by the whole workgroup, once row-major and once transposed where an
//   operand needs the token dimension as its contraction dimension.
// * Softmax runs in the log2 domain with an online max over key tiles; the
//   bias table of one head lives in LDS (pre-scaled by log2 e) and the mask
//   is a label compare per pair.
// * The bias-table gradient is summed per workgroup in LDS (one head per
//   workgroup, many windows per workgroup), written as per-workgroup
//   partials, and reduced in a fixed order by a second kernel.
#include "terra_common.h"

namespace terra {

// Window-resident path (attn_win.hip) for windows of at most 128 tokens.
bool win_fwd_ok(const Geo& g, bool bf16_);
bool win_bwd_ok(const Geo& g, bool bf16_);
int win_bwd_nslice(const Geo& g);
size_t win_fwd_lds(const Geo& g);
size_t win_bwd_lds(const Geo& g);
hipError_t launch_win_fwd(const Geo& g, bool nhwc, const void* q, const void* k, const void* v,
                          const float* table, void* o, float* lse, hipStream_t st);
hipError_t launch_win_bwd(const Geo& g, bool nhwc, const void* q, const void* k, const void* v,
                          const void* dout, const float* lse, const float* table, void* dq,
                          void* dk, void* dv, float* partial, int nslice, hipStream_t st);
// Fixed-order sum of the per-slice bias-gradient partials (dtab.hip).
hipError_t launch_dtab_reduce(const Geo& g, const float* partial, float* dtab, int nslice,
                              hipStream_t st);

constexpr int kThreads = 256;   // 4 waves
constexpr int kWaveQ = 32;      // queries (or keys) per wave
constexpr int kChunk = 128;     // queries (or keys) per workgroup
// Keys (or queries) per LDS tile: 64, or 32 for fp32 with head_dim 64 or 128
// (so that a staged tile set stays within 80 KB of LDS).
template <typename T, int HD> constexpr int tile_of() { return (sizeof(T) == 4 && HD >= 64) ? 32 : 64; }
constexpr int kPad = 8;         // LDS row padding, elements
constexpr int kLabBad = 0xFF;   // label of padding slots (never matches)

// Work item of a forward workgroup.  The hardware hands consecutive
// workgroups to the 8 XCDs in turn; giving each XCD one contiguous range of
// items puts the query chunks of one window and head, which stage the same
// K/V tiles, behind the same L2 (forward -2 to -4 %; measured no better or
// slower for the dK/dV and dQ kernels, which keep the plain order).  The grid
// is rounded up to a multiple of 8 and the padding workgroups exit at once.
__device__ inline int xcd_item(int bid, int nblocks) { return (bid & 7) * (nblocks >> 3) + (bid >> 3); }
static inline int grid8(int n) { return (n + 7) & ~7; }

// Transposed tiles (head-dim rows e, token columns): row e starts at
// e * (kTile + kPad) plus 4 elements per group of 8 rows, so that the
// transposing staging stores of one instruction (8 rows of one chunk, the
// chunks 8 rows apart) fall in distinct LDS banks.
template <typename T, int HD>
__device__ __host__ constexpr int tr_row(int e) { return e * (tile_of<T, HD>() + kPad) + (e >> 3) * 4; }
template <typename T, int HD>
__device__ __host__ constexpr int tr_size() { return tr_row<T, HD>(HD); }

// 16-bit V tiles stay row-major and give their transposed operands through
// the LDS transpose read: in each 16-lane group G of that read, lane i
// receives element i % 4 of the 8 bytes addressed by lane 16 G + 4 x + i / 4,
// x = 0..3.  Row stride 16 mod 64 dwords, so the 4 rows x 64 bytes of two
// groups fall in distinct LDS banks.
template <int HD> constexpr int tr16_stride() { return HD == 32 ? 32 : HD == 64 ? 96 : 160; }
template <typename T, int HD>
__device__ __host__ constexpr int vtile_size() {
  return sizeof(T) == 2 ? tile_of<T, HD>() * tr16_stride<HD>() : tr_size<T, HD>();
}
// Transposed copy of a tile: needed for fp32 only (16-bit tiles are read
// transposed straight from their row-major copy).
template <typename T, int HD>
__device__ __host__ constexpr int ttile_size() { return sizeof(T) == 2 ? 0 : tr_size<T, HD>(); }

// Slot s (0..7) of lane half h inside a 16-deep contraction chunk, when the
// operand comes from 32x32 result registers 8c..8c+7: row acc_row(s, h).
__device__ inline int perm_slot(int s, int h) { return 8 * (s / 4) + 4 * h + (s % 4); }

template <typename T>
__device__ inline typename Operand<T>::type load_op_global(const T* p) {
  return *reinterpret_cast<const typename Operand<T>::type*>(p);
}
template <typename T>
__device__ inline typename Operand<T>::type zero_op() {
  typename Operand<T>::type z;
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = from_float<T>(0.0f);
  return z;
}
// Operand from an LDS row, 8 consecutive elements.
template <typename T>
__device__ inline typename Operand<T>::type load_op_lds(const T* p) {
  return *reinterpret_cast<const typename Operand<T>::type*>(p);
}
// Operand from an LDS row in the permuted slot order (two runs of 4).
template <typename T>
__device__ inline typename Operand<T>::type load_op_lds_perm(const T* row, int h) {
  typename Operand<T>::type o;
  const T* p0 = row + 4 * h;
  const T* p1 = row + 8 + 4 * h;
#pragma unroll
  for (int s = 0; s < 4; ++s) { o[s] = p0[s]; o[4 + s] = p1[s]; }
  return o;
}

// One staged tile of one tensor held in registers between its load from HBM
// and its store to LDS, so that the next tile's loads overlap the current
// tile's matrix work: thread t holds 16-byte chunks t, t+256, ... (row =
// chunk / chunks-per-row).
template <typename T, int HD>
struct TileRegs {
  static constexpr int kCpr = HD * (int)sizeof(T) / 16;
  static constexpr int kPer = tile_of<T, HD>() * kCpr / kThreads;
  uint4 r[kPer];
};

template <typename T, int HD, bool NHWC>
__device__ inline void tile_load(TileRegs<T, HD>& t, const T* __restrict__ src, const Geo& g,
                                 const WinTokens<NHWC>& wt, int r0, int n, int hoff) {
  constexpr int kCpr = TileRegs<T, HD>::kCpr;
#pragma unroll
  for (int u = 0; u < TileRegs<T, HD>::kPer; ++u) {
    const int idx = threadIdx.x + u * kThreads;
    const int rr = idx / kCpr, ch = idx % kCpr;
    const int row = r0 + rr;
    t.r[u] = make_uint4(0, 0, 0, 0);
    if (row < n)
      t.r[u] = *reinterpret_cast<const uint4*>(src + wt.tok(g, row) * g.C + hoff + ch * (16 / (int)sizeof(T)));
  }
}

// Element offsets (token index times C) of the window's n tokens, so that
// the staging of each later tile reads its row addresses from LDS instead of
// redoing the shifted-coordinate arithmetic per chunk (fused route only;
// window-major rows are consecutive).  The writes become visible to the
// other waves at the next barrier; the first tile is staged from its own
// arithmetic.
template <bool NHWC>
__device__ inline void tok_fill(uint32_t* tt, const Geo& g, const WinTokens<NHWC>& wt, int n) {
  if constexpr (NHWC)
    for (int t = threadIdx.x; t < n; t += kThreads) tt[t] = wt.tok(g, t) * (uint32_t)g.C;
}

// tile_load with the row offsets taken from the table.
template <typename T, int HD, bool NHWC>
__device__ inline void tile_load_tt(TileRegs<T, HD>& t, const T* __restrict__ src, const Geo& g,
                                    const WinTokens<NHWC>& wt, const uint32_t* tt, int r0, int n,
                                    int hoff) {
  if constexpr (!NHWC) {
    tile_load(t, src, g, wt, r0, n, hoff);
  } else {
    constexpr int kCpr = TileRegs<T, HD>::kCpr;
#pragma unroll
    for (int u = 0; u < TileRegs<T, HD>::kPer; ++u) {
      const int idx = threadIdx.x + u * kThreads;
      const int rr = idx / kCpr, ch = idx % kCpr;
      const int row = r0 + rr;
      t.r[u] = make_uint4(0, 0, 0, 0);
      if (row < n)
        t.r[u] = *reinterpret_cast<const uint4*>(src + tt[row] + hoff + ch * (16 / (int)sizeof(T)));
    }
  }
}

// Row-major store of a staged tile with row stride RS elements.
template <typename T, int HD, int RS>
__device__ inline void tile_store_rows(const TileRegs<T, HD>& t, T* lds) {
  constexpr int kCpr = TileRegs<T, HD>::kCpr;
#pragma unroll
  for (int u = 0; u < TileRegs<T, HD>::kPer; ++u) {
    const int idx = threadIdx.x + u * kThreads;
    const int rr = idx / kCpr, ch = idx % kCpr;
    *reinterpret_cast<uint4*>(lds + rr * RS + ch * (16 / (int)sizeof(T))) = t.r[u];
  }
}

template <typename T, int HD, bool ROWMAJOR, bool TRANS>
__device__ inline void tile_store(const TileRegs<T, HD>& t, T* lds_rm, T* lds_tr) {
  constexpr int kCpr = TileRegs<T, HD>::kCpr;
  constexpr int kElemPerChunk = 16 / sizeof(T);
#pragma unroll
  for (int u = 0; u < TileRegs<T, HD>::kPer; ++u) {
    const int idx = threadIdx.x + u * kThreads;
    const int rr = idx / kCpr, ch = idx % kCpr;
    if (ROWMAJOR) *reinterpret_cast<uint4*>(lds_rm + rr * (HD + kPad) + ch * kElemPerChunk) = t.r[u];
    if (TRANS) {
      const T* e = reinterpret_cast<const T*>(&t.r[u]);
#pragma unroll
      for (int x = 0; x < kElemPerChunk; ++x) lds_tr[tr_row<T, HD>(ch * kElemPerChunk + x) + rr] = e[x];
    }
  }
}

// Label/bias-offset word of in-window token t (t < n), or of a pad slot.
__device__ inline int token_info(const Geo& g, int i, int j, int cols, int t, int n) {
  if (t >= n) return kLabBad << 24;
  const int a = fast_div(t, cols, win_rcols(g, j));
  const int c = t - a * cols;
  const int lab = row_label(g, i * g.wh + a) | col_label(g, j * g.ww + c);
  return (a * g.bstride + c) | (lab << 24);
}

// bias_init with each key's bias offset also held as a byte offset, knb[k]
// = 4 x (offset of key k): one group of four keys then costs one address add
// from tabq, the lane's row of the reversed table in bytes.  Labels still
// come from kinfo, and an excluded pair reads its bin (always inside the
// table) and is replaced by -inf.
template <bool QUAD, bool MASK>
__device__ inline f32x16 bias_init_nb(const int* kinfo, const int* knb, const char* tabq, int kb,
                                      int half, int qlab) {
  f32x16 c;
#pragma unroll
  for (int g4 = 0; g4 < 4; ++g4) {
    const int kk = 32 * kb + 8 * g4 + 4 * half;
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const int kx = QUAD ? kk : kk + x;
      c[4 * g4 + x] = reinterpret_cast<const float*>(tabq + knb[kx])[QUAD ? x : 0];
      if (MASK && (kinfo[kx] >> 24) != qlab) c[4 * g4 + x] = -INFINITY;
    }
  }
  return c;
}

// The key-major form (lane = key, registers = queries of query block QB):
// qnb[t] = 4 x (offset of query t), tabk the lane's row of the forward-order
// table in bytes.
template <bool QUAD, bool MASK>
__device__ inline f32x16 bias_init_t_nb(const int* qinfo, const int* qnb, const char* tabk, int qb,
                                        int half, int klab) {
  f32x16 c;
#pragma unroll
  for (int g4 = 0; g4 < 4; ++g4) {
    const int qq = 32 * qb + 8 * g4 + 4 * half;
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const int qx = QUAD ? qq : qq + x;
      c[4 * g4 + x] = reinterpret_cast<const float*>(tabk + qnb[qx])[QUAD ? x : 0];
      if (MASK && (qinfo[qx] >> 24) != klab) c[4 * g4 + x] = -INFINITY;
    }
  }
  return c;
}

// ---------------------------------------------------------------------------
// Forward.  Grid: B * nwin * heads * nqc workgroups (nqc query chunks of 128
// per window, empty chunks of small windows exit at once).  The bias enters
// the score accumulator before the QK^T product (table times sqrt(hd) in
// reversed bin order, -inf entries for excluded pairs), so each score costs
// one multiply-add and one exp2 outside the matrix cores.  With olo (16-bit
// types, nullable) the PV product also takes P's rounding residual and the
// epilogue writes O's: the backward's D = <dO, O> then needs no key sweep.
// ---------------------------------------------------------------------------
template <typename T, int HD, bool NHWC, bool QUAD, bool SPLIT>
__global__ __launch_bounds__(kThreads) void fwd_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const float* __restrict__ table, T* __restrict__ o, T* __restrict__ olo,
    float* __restrict__ lse, Geo g, int nqc, float scale_log2) {
  constexpr int kTile = tile_of<T, HD>();
  extern __shared__ __align__(16) char smem[];
  T* kt = reinterpret_cast<T*>(smem);                          // [kTile][HD+kPad]
  T* vt = kt + kTile * (HD + kPad);                            // V^T, or V rows (16-bit)
  int* kinfo = reinterpret_cast<int*>(vt + vtile_size<T, HD>());
  float* tab = reinterpret_cast<float*>(kinfo + kTile);        // [nbins+4], reversed
  uint32_t* tt = reinterpret_cast<uint32_t*>(tab + g.nbins + 4);   // [wh*ww] token offsets

  int bid = xcd_item(blockIdx.x, gridDim.x);
  if (bid >= g.B * g.nwin * g.heads * nqc) return;
  const int qc = bid % nqc; bid /= nqc;
  const int h = bid % g.heads; bid /= g.heads;
  const int w = bid % g.nwin;
  const int b = bid / g.nwin;
  const int i = w / g.Mw, j = w - (w / g.Mw) * g.Mw;
  const int cols = win_cols(g, j);
  const int n = win_rows(g, i) * cols;
  const int q0 = qc * kChunk;
  if (q0 >= n) return;
  const WinTokens<NHWC> wt(g, b, i, j);
  const int hoff = h * HD;

  const float bscale = sqrtf((float)HD);
  for (int x = threadIdx.x; x < g.nbins + 4; x += kThreads)
    tab[x] = x < g.nbins ? table[(g.nbins - 1 - x) * g.heads + h] * bscale : -INFINITY;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int qi = q0 + wave * kWaveQ + col;
  const bool qvalid = qi < n;
  // waves whose 32 queries all lie past the window's end (last chunk of a
  // window that is not a multiple of 128 tokens) skip the matrix work
  const bool wactive = q0 + wave * kWaveQ < n;
  const int qinf = token_info(g, i, j, cols, qvalid ? qi : 0, n);
  const int qlab = qinf >> 24;
  const int qrev = g.nbins - 1 - ((qinf & 0xFFFFFF) + (g.wh - 1) * g.bstride + (g.ww - 1));
  const bool mask = window_has_labels(g, i, j) || (n % kTile) != 0;
  constexpr bool split = SPLIT && sizeof(T) == 2;

  typename Operand<T>::type qop[HD / 16];
#pragma unroll
  for (int c = 0; c < HD / 16; ++c)
    qop[c] = qvalid ? load_op_global<T>(q + wt.tok(g, qi) * g.C + hoff + 16 * c + 8 * half)
                    : zero_op<T>();

  f32x16 oacc[HD / 32];
#pragma unroll
  for (int eb = 0; eb < HD / 32; ++eb) oacc[eb] = f32x16{};
  float m_run = -1e30f, l_run = 0.0f;     // running max (log2 units) and sum
  constexpr float kPOff = __is_same(T, _Float16) ? 7.0f : 0.0f;

  // K, V tiles go HBM -> registers -> LDS, one tile ahead up to head dim 64
  constexpr bool kPrefetch = HD <= 64;
  TileRegs<T, HD> rk, rv;
  if (kPrefetch) {
    tile_load(rk, k, g, wt, 0, n, hoff);
    tile_load(rv, v, g, wt, 0, n, hoff);
  }
  tok_fill(tt, g, wt, n);
  if (!kPrefetch && NHWC) lds_barrier();   // the first tile comes from the table too
  for (int k0 = 0; k0 < n; k0 += kTile) {
    if (!kPrefetch) {
      tile_load_tt(rk, k, g, wt, tt, k0, n, hoff);
      tile_load_tt(rv, v, g, wt, tt, k0, n, hoff);
    }
    lds_barrier();
    tile_store<T, HD, true, false>(rk, kt, nullptr);
    if (sizeof(T) == 2) tile_store_rows<T, HD, tr16_stride<HD>()>(rv, vt);
    else tile_store<T, HD, false, true>(rv, nullptr, vt);
    if (threadIdx.x < kTile) kinfo[threadIdx.x] = token_info(g, i, j, cols, k0 + threadIdx.x, n);
    lds_barrier();
    if (kPrefetch && k0 + kTile < n) {
      tile_load_tt(rk, k, g, wt, tt, k0 + kTile, n, hoff);
      tile_load_tt(rv, v, g, wt, tt, k0 + kTile, n, hoff);
    }
    if (!wactive) continue;     // staging and barriers only

    f32x16 s[kTile / 32];
    float mloc = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < kTile / 32; ++kb) {
      s[kb] = mask ? bias_init<QUAD, true>(kinfo, tab, kb, half, qrev, qlab, g.nbins)
                   : bias_init<QUAD, false>(kinfo, tab, kb, half, qrev, qlab, g.nbins);
#pragma unroll
      for (int c = 0; c < HD / 16; ++c)
        mma16(s[kb], load_op_lds<T>(kt + (kb * 32 + col) * (HD + kPad) + 16 * c + 8 * half), qop[c]);
#pragma unroll
      for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, s[kb][r]);
    }
    mloc = halves_max(mloc);
    // The running maximum moves (and O and the sum are rescaled) only when
    // some query of the wave sees a score more than 2^8 above it: between
    // moves the weights stay below 256, which the fp32 sums and the 16-bit
    // operands carry as exactly as weights below 1.  For float16 operands
    // the weights run 2^kPOff higher (m_run sits kPOff below the maximum;
    // the sum, and so the LSE, follow), so that weights down to 2^-21 of the
    // maximum, and the low parts of the split, stay above float16's
    // subnormal range (6.1e-5), which the operands would lose.
    const float mt = mloc * scale_log2;
    if (__builtin_amdgcn_ballot_w64(mt > m_run + (kPOff + 8.0f)) != 0) {
      const float mnew = fmaxf(m_run, mt - kPOff);
      const float alpha = exp2f(m_run - mnew);
      m_run = mnew;
      l_run *= alpha;
#pragma unroll
      for (int eb = 0; eb < HD / 32; ++eb) oacc[eb] *= alpha;
    }
#pragma unroll
    for (int kb = 0; kb < kTile / 32; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(s[kb][r] * scale_log2 - m_run);
        s[kb][r] = p;
        l_run += p;
      }
    }
    if constexpr (sizeof(T) == 2) {
      // 16-bit P operands.  When the caller keeps O_lo, P also enters as
      // hi + lo (lo = P - hi rounded again), so that the fp32 sum carries
      // P V to about 16 significant bits rather than the 8 of one rounding.
      typename Operand<T>::type phi[kTile / 32][2], plo[kTile / 32][2];
#pragma unroll
      for (int kb = 0; kb < kTile / 32; ++kb)
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          phi[kb][c] = pack8<T>(s[kb], 8 * c);
          if constexpr (split) {
#pragma unroll
            for (int x = 0; x < 8; ++x)
              plo[kb][c][x] = from_float<T>(s[kb][8 * c + x] - to_float<T>(phi[kb][c][x]));
          }
        }
#pragma unroll
      for (int eb = 0; eb < HD / 32; ++eb) {
#pragma unroll
        for (int kb = 0; kb < kTile / 32; ++kb) {
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            const auto vop = lds_tr_op<T, tr16_stride<HD>()>(vt, kb, c, eb, lane);
            mma16(oacc[eb], vop, phi[kb][c]);
            if constexpr (split) mma16(oacc[eb], vop, plo[kb][c]);
          }
        }
      }
    } else {
#pragma unroll
      for (int eb = 0; eb < HD / 32; ++eb) {
#pragma unroll
        for (int kb = 0; kb < kTile / 32; ++kb) {
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            const T* row = vt + tr_row<T, HD>(eb * 32 + col) + kb * 32 + 16 * c;
            mma16(oacc[eb], load_op_lds_perm<T>(row, half), pack8<T>(s[kb], 8 * c));
          }
        }
      }
    }
  }
  l_run = halves_sum(l_run);
  if (!qvalid) return;
  const float inv = 1.0f / l_run;
  T* orow = o + wt.tok(g, qi) * g.C + hoff;
  // O_lo: what rounding O to T left out, itself rounded to T; O + O_lo
  // carries the fp32 output to about 16 significant bits
  T* lrow = split ? olo + wt.tok(g, qi) * g.C + hoff : nullptr;
  const unsigned opq = (unsigned)g.C >> 31;    // 0: C is positive
  (void)lrow;
  (void)opq;
#pragma unroll
  for (int eb = 0; eb < HD / 32; ++eb) {
#pragma unroll
    for (int grp = 0; grp < 4; ++grp) {
      const int e = eb * 32 + 8 * grp + 4 * half;
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        float val = oacc[eb][4 * grp + x] * inv;
        // The split needs one float32 value behind both halves: left to
        // itself the compiler folds the multiply into a float16
        // mixed-precision multiply on the O_lo side (one rounding of
        // acc * inv) while the stored O rounds the float32 product again,
        // and near a tie the two pick different halves.  OR-ing in a zero
        // the compiler cannot prove (opq) stops that fold.  (An empty asm
        // register barrier did too, but slowed the whole kernel by half.)
        if constexpr (split) val = __uint_as_float(__float_as_uint(val) | opq);
        const T hi = from_float<T>(val);
        orow[e + x] = hi;
        if constexpr (split) lrow[e + x] = from_float<T>(val - to_float<T>(hi));
      }
    }
  }
  if (half == 0) lse[wt.lse_at(g, h, qi)] = (m_run + __log2f(l_run)) * kLn2;
}

// ---------------------------------------------------------------------------
// Backward, step 1: D, dQ and the bias-table partials.  One head per
// workgroup; the workgroup walks items (image, window, query chunk)
// slice, slice + nslice, ... in a fixed order and accumulates dT in LDS.
// Per item, D_q = sum_k P dP = <dO_q, O_q> (O unrounded) is formed first
// and stored for the dK/dV kernel: from the forward's O and its rounding
// residual O_lo when the caller kept it (olo not null), else by a first
// sweep over the key tiles in fp32.  The stored 16-bit O alone is not
// enough: D's rounding error, alike for every key of a query, adds up over
// the windows in the bias-table gradient.  The (second) sweep forms dS, dQ
// and the bias bins.
// ---------------------------------------------------------------------------
template <typename T, int HD, bool NHWC, bool QUAD, bool RES>
__global__ __launch_bounds__(kThreads, 2) void bwd_dq_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const T* __restrict__ o, const T* __restrict__ olo,
    const T* __restrict__ dout, const float* __restrict__ lse, float* __restrict__ D,
    const float* __restrict__ table, T* __restrict__ dq, float* __restrict__ partial,
    Geo g, int nqc, int nslice, float scale_log2, float scale) {
  constexpr int kTile = tile_of<T, HD>();
  constexpr int kTE = kTile * (HD + kPad);            // elements of one staged tile
  // RES: every tile of the window stays in LDS for the whole item (nt tiles)
  const int nt = RES ? (g.wh * g.ww + kTile - 1) / kTile : 1;
  extern __shared__ __align__(16) char smem[];
  T* kt0 = reinterpret_cast<T*>(smem);                // K  nt x [kTile][HD+kPad]
  T* vr0 = kt0 + nt * kTE;                            // V  nt x [kTile][HD+kPad]
  T* ktt = vr0 + nt * kTE;                            // K^T (transposed tile, fp32)
  // nt x {[kTile] label/offset words, [kTile] 4 x offset}
  int* kinfo0 = reinterpret_cast<int*>(ktt + ttile_size<T, HD>());
  float* tab = reinterpret_cast<float*>(kinfo0 + 2 * nt * kTile);   // [nbins+4], reversed
  float* dtab = tab + g.nbins + 4;                    // [4][nbins], one per wave
  // [wh*ww] token offsets of the current item.  One buffer serves: the last
  // read of an item (the prefetch of its last tile) comes before the
  // barriers of that tile, which every wave passes before the next fill.
  uint32_t* tt = reinterpret_cast<uint32_t*>(dtab + 4 * g.nbins);

  const int h = blockIdx.x / nslice;
  const int slice = blockIdx.x - h * nslice;
  const int hoff = h * HD;
  const float bscale = sqrtf((float)HD);
  for (int x = threadIdx.x; x < g.nbins + 4; x += kThreads)
    tab[x] = x < g.nbins ? table[(g.nbins - 1 - x) * g.heads + h] * bscale : -INFINITY;
  for (int x = threadIdx.x; x < 4 * g.nbins; x += kThreads) dtab[x] = 0.0f;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int nitems = g.B * g.nwin * nqc;

  for (int it = slice; it < nitems; it += nslice) {
    const int qc = it % nqc;
    const int w = (it / nqc) % g.nwin;
    const int b = it / (nqc * g.nwin);
    const int i = w / g.Mw, j = w - (w / g.Mw) * g.Mw;
    const int cols = win_cols(g, j);
    const int n = win_rows(g, i) * cols;
    const int q0 = qc * kChunk;
    if (q0 >= n) continue;
    const WinTokens<NHWC> wt(g, b, i, j);
    const int qi = q0 + wave * kWaveQ + col;
    const bool qvalid = qi < n;
    const bool wactive = q0 + wave * kWaveQ < n;   // else staging and barriers only
    const int qinf = token_info(g, i, j, cols, qvalid ? qi : 0, n);
    const int qlab = qinf >> 24;
    const int qoff = (qinf & 0xFFFFFF) + (g.wh - 1) * g.bstride + (g.ww - 1);
    const int qrev = g.nbins - 1 - qoff;
    const char* tabq = reinterpret_cast<const char*>(tab + qrev);
    const int64_t lidx = wt.lse_at(g, h, qvalid ? qi : 0);
    // +inf for padding queries: their P is exactly 0
    const float lse2 = qvalid ? lse[lidx] * kLog2e : INFINITY;
    const bool mask = window_has_labels(g, i, j) || (n % kTile) != 0;

    typename Operand<T>::type qop[HD / 16], dop[HD / 16];
#pragma unroll
    for (int c = 0; c < HD / 16; ++c) {
      qop[c] = qvalid ? load_op_global<T>(q + wt.tok(g, qi) * g.C + hoff + 16 * c + 8 * half)
                      : zero_op<T>();
      dop[c] = qvalid ? load_op_global<T>(dout + wt.tok(g, qi) * g.C + hoff + 16 * c + 8 * half)
                      : zero_op<T>();
    }
    // D_q, then the sweep.  The K, V tiles go HBM -> registers -> LDS; up to
    // head dim 64 each tile's loads are issued while the previous tile
    // computes (after the last tile of the D sweep, or straight after these
    // first loads when D comes from O, come the first tiles of the main
    // sweep); at head dim 128 the registers this holds would halve the
    // occupancy.
    constexpr bool kPrefetch = HD <= 64;
    TileRegs<T, HD> rk, rv;
    if constexpr (RES) {
      // all tiles of the window into LDS once per item (each tile's loads
      // issued before the previous tile is stored); both sweeps then read
      // them without staging or barriers
      tile_load(rk, k, g, wt, 0, n, hoff);
      tile_load(rv, v, g, wt, 0, n, hoff);
      lds_barrier();                  // the previous item is done with the tiles
      for (int t0 = 0; t0 < n; t0 += kTile) {
        TileRegs<T, HD> nk = rk, nv = rv;
        if (t0 + kTile < n) {
          tile_load(nk, k, g, wt, t0 + kTile, n, hoff);
          tile_load(nv, v, g, wt, t0 + kTile, n, hoff);
        }
        const int tix = t0 / kTile;
        tile_store<T, HD, true, false>(rk, kt0 + tix * kTE, nullptr);
        tile_store<T, HD, true, false>(rv, vr0 + tix * kTE, nullptr);
        if (threadIdx.x < kTile) {
          const int inf = token_info(g, i, j, cols, t0 + threadIdx.x, n);
          kinfo0[tix * 2 * kTile + threadIdx.x] = inf;
          kinfo0[tix * 2 * kTile + kTile + threadIdx.x] = 4 * (inf & 0xFFFFFF);
        }
        rk = nk;
        rv = nv;
      }
      lds_barrier();
    } else if (kPrefetch) {
      tile_load(rk, k, g, wt, 0, n, hoff);
      tile_load(rv, v, g, wt, 0, n, hoff);
    }
    if constexpr (!RES) {
      tok_fill(tt, g, wt, n);
      if (!kPrefetch && NHWC) lds_barrier();   // the first tile comes from the table too
    }
    float dsum = 0.0f;
    if (olo != nullptr) {
      // D from the forward's output: the two halves of a lane pair hold
      // alternate 8-element runs of the query's row, like dop
      if (qvalid) {
        const T* orow = o + wt.tok(g, qi) * g.C + hoff;
        const T* lrow = olo + wt.tok(g, qi) * g.C + hoff;
#pragma unroll
        for (int c = 0; c < HD / 16; ++c) {
          const auto ov = load_op_global<T>(orow + 16 * c + 8 * half);
          const auto lv = load_op_global<T>(lrow + 16 * c + 8 * half);
#pragma unroll
          for (int x = 0; x < 8; ++x)
            dsum += to_float<T>(dop[c][x]) * (to_float<T>(ov[x]) + to_float<T>(lv[x]));
        }
      }
    } else for (int k0 = 0; k0 < n; k0 += kTile) {
      const int tix = RES ? k0 / kTile : 0;
      T* kt = kt0 + tix * kTE;
      T* vr = vr0 + tix * kTE;
      int* kinfo = kinfo0 + tix * 2 * kTile;
      int* knb = kinfo + kTile;
      if constexpr (!RES) {
        if (!kPrefetch) {
          tile_load_tt(rk, k, g, wt, tt, k0, n, hoff);
          tile_load_tt(rv, v, g, wt, tt, k0, n, hoff);
        }
        lds_barrier();
        tile_store<T, HD, true, false>(rk, kt, nullptr);
        tile_store<T, HD, true, false>(rv, vr, nullptr);
        if (threadIdx.x < kTile) {
          const int inf = token_info(g, i, j, cols, k0 + threadIdx.x, n);
          kinfo[threadIdx.x] = inf;
          knb[threadIdx.x] = 4 * (inf & 0xFFFFFF);
        }
        lds_barrier();
        if (kPrefetch) {
          const int nk0 = k0 + kTile < n ? k0 + kTile : 0;
          tile_load_tt(rk, k, g, wt, tt, nk0, n, hoff);
          tile_load_tt(rv, v, g, wt, tt, nk0, n, hoff);
        }
      }
      if (!wactive) continue;
#pragma unroll
      for (int kb = 0; kb < kTile / 32; ++kb) {
        f32x16 s = mask ? bias_init_nb<QUAD, true>(kinfo, knb, tabq, kb, half, qlab)
                        : bias_init_nb<QUAD, false>(kinfo, knb, tabq, kb, half, qlab);
        f32x16 dp = f32x16{};
#pragma unroll
        for (int c = 0; c < HD / 16; ++c) {
          mma16(s, load_op_lds<T>(kt + (kb * 32 + col) * (HD + kPad) + 16 * c + 8 * half), qop[c]);
          mma16(dp, load_op_lds<T>(vr + (kb * 32 + col) * (HD + kPad) + 16 * c + 8 * half), dop[c]);
        }
#pragma unroll
        for (int r = 0; r < 16; ++r)
          dsum += __builtin_amdgcn_exp2f(s[r] * scale_log2 - lse2) * dp[r];
      }
    }
    const float Dq = halves_sum(dsum);
    if (qvalid && half == 0) D[lidx] = Dq;

    // main sweep: dS, dQ, bias bins
    const bool fold = (g.ww % 4 == 0) && (g.W % g.ww) % 4 == 0;   // uniform
    const int cq = qi - fast_div(qi, cols, win_rcols(g, j)) * cols;
    // runs: lanes of one 32-lane half holding consecutive queries of one
    // window row; run = lanes before this one in its run, rest = lanes after
    const int run = cq < col ? cq : col;
    const int rest = (cols - 1 - cq) < (31 - col) ? (cols - 1 - cq) : (31 - col);
    const float fnext = rest > 0 ? 1.0f : 0.0f;          // lane l+1 is in the run
    const float fsend = fnext;                           // this lane may pass to l+1
    const float fkeep = run < 3 ? 1.0f : 0.0f;           // one of the run's first three
    f32x16 dqacc[HD / 32];
#pragma unroll
    for (int eb = 0; eb < HD / 32; ++eb) dqacc[eb] = f32x16{};

    for (int k0 = 0; k0 < n; k0 += kTile) {
      const int tix = RES ? k0 / kTile : 0;
      T* kt = kt0 + tix * kTE;
      T* vr = vr0 + tix * kTE;
      int* kinfo = kinfo0 + tix * 2 * kTile;
      int* knb = kinfo + kTile;
      if constexpr (!RES) {
        if (!kPrefetch) {
          tile_load_tt(rk, k, g, wt, tt, k0, n, hoff);
          tile_load_tt(rv, v, g, wt, tt, k0, n, hoff);
        }
        lds_barrier();
        tile_store<T, HD, true, sizeof(T) == 4>(rk, kt, ktt);
        tile_store<T, HD, true, false>(rv, vr, nullptr);
        if (threadIdx.x < kTile) {
          const int inf = token_info(g, i, j, cols, k0 + threadIdx.x, n);
          kinfo[threadIdx.x] = inf;
          knb[threadIdx.x] = 4 * (inf & 0xFFFFFF);
        }
        lds_barrier();
        if (kPrefetch && k0 + kTile < n) {
          tile_load_tt(rk, k, g, wt, tt, k0 + kTile, n, hoff);
          tile_load_tt(rv, v, g, wt, tt, k0 + kTile, n, hoff);
        }
      }
      if (!wactive) continue;
      // Head dim 64: the S and dP products of every key block of the tile
      // first, then per block dS and dQ += dS K, so that one block's exp
      // runs while the next block's products are on the matrix cores; each
      // block's K and V operands are read from LDS before its bias (dQ
      // kernel -3 % at 576-token windows).  Otherwise one block at a time:
      // at head dim 128 the held operands and accumulators would spill, and
      // at head dim 32 they would cost the third resident wave per SIMD.
      constexpr bool kHold = HD == 64;
      f32x16 dsb[kTile / 32];
      if constexpr (kHold) {
        f32x16 sb[kTile / 32];
#pragma unroll
        for (int kb = 0; kb < kTile / 32; ++kb) {
          typename Operand<T>::type kop_[HD / 16], vop_[HD / 16];
#pragma unroll
          for (int c = 0; c < HD / 16; ++c) {
            kop_[c] = load_op_lds<T>(kt + (kb * 32 + col) * (HD + kPad) + 16 * c + 8 * half);
            vop_[c] = load_op_lds<T>(vr + (kb * 32 + col) * (HD + kPad) + 16 * c + 8 * half);
          }
          __builtin_amdgcn_sched_barrier(0);
          sb[kb] = mask ? bias_init_nb<QUAD, true>(kinfo, knb, tabq, kb, half, qlab)
                        : bias_init_nb<QUAD, false>(kinfo, knb, tabq, kb, half, qlab);
#pragma unroll
          for (int r = 0; r < 16; ++r) dsb[kb][r] = -Dq;      // dP - D straight from the product
#pragma unroll
          for (int c = 0; c < HD / 16; ++c) {
            mma16(sb[kb], kop_[c], qop[c]);
            mma16(dsb[kb], vop_[c], dop[c]);
          }
        }
#pragma unroll
        for (int kb = 0; kb < kTile / 32; ++kb) {
#pragma unroll
          for (int r = 0; r < 16; ++r) dsb[kb][r] *= __builtin_amdgcn_exp2f(sb[kb][r] * scale_log2 - lse2);
#pragma unroll
          for (int eb = 0; eb < HD / 32; ++eb) {
#pragma unroll
            for (int c = 0; c < 2; ++c) {
              if constexpr (sizeof(T) == 2) {
                mma16(dqacc[eb], lds_tr_op<T, HD + kPad>(kt, kb, c, eb, lane), pack8<T>(dsb[kb], 8 * c));
              } else {
                const T* row = ktt + tr_row<T, HD>(eb * 32 + col) + kb * 32 + 16 * c;
                mma16(dqacc[eb], load_op_lds_perm<T>(row, half), pack8<T>(dsb[kb], 8 * c));
              }
            }
          }
        }
      } else {
#pragma unroll
        for (int kb = 0; kb < kTile / 32; ++kb) {
          f32x16 s = mask ? bias_init_nb<QUAD, true>(kinfo, knb, tabq, kb, half, qlab)
                          : bias_init_nb<QUAD, false>(kinfo, knb, tabq, kb, half, qlab);
          f32x16 dp;
#pragma unroll
          for (int r = 0; r < 16; ++r) dp[r] = -Dq;      // dP - D straight from the product
#pragma unroll
          for (int c = 0; c < HD / 16; ++c) {
            mma16(s, load_op_lds<T>(kt + (kb * 32 + col) * (HD + kPad) + 16 * c + 8 * half), qop[c]);
            mma16(dp, load_op_lds<T>(vr + (kb * 32 + col) * (HD + kPad) + 16 * c + 8 * half), dop[c]);
          }
#pragma unroll
          for (int r = 0; r < 16; ++r) dsb[kb][r] = __builtin_amdgcn_exp2f(s[r] * scale_log2 - lse2) * dp[r];
#pragma unroll
          for (int eb = 0; eb < HD / 32; ++eb) {
#pragma unroll
            for (int c = 0; c < 2; ++c) {
              if constexpr (sizeof(T) == 2) {
                mma16(dqacc[eb], lds_tr_op<T, HD + kPad>(kt, kb, c, eb, lane), pack8<T>(dsb[kb], 8 * c));
              } else {
                const T* row = ktt + tr_row<T, HD>(eb * 32 + col) + kb * 32 + 16 * c;
                mma16(dqacc[eb], load_op_lds_perm<T>(row, half), pack8<T>(dsb[kb], 8 * c));
              }
            }
          }
        }
      }
      // Bias bins: each wave adds into its own copy, and the two lane halves
      // add with separate instructions.  Within one half, lanes hold distinct
      // queries of the same key, hence distinct bins, so the additions are
      // plain read-modify-writes (an LDS float atomic costs about three
      // clocks per lane, some 170 times a store) and every bin receives them
      // in program order; lanes with nothing to add (padding queries,
      // excluded pairs) stay out.  When every window width is a
      // multiple of 4, registers 4g..4g+3 hold four consecutive keys k..k+3
      // of one window row and (q, k+x), (q+1, k+x+1) share a bin.  Within a
      // run of consecutive lanes holding consecutive queries of one window
      // row, a DPP chain towards lower lanes folds each group into one value
      // (bin of (q, k)); the pairs it cannot reach (fewer than x lanes
      // before q in the run) move towards higher lanes into the run's first
      // three lanes (bin of (q', k+3)), and the few that would leave a run
      // shorter than three lanes are added on their own.
      float* mybins = dtab + wave * g.nbins;
      // bin of (this lane's query, key kk): qbins - knb[kk] in bytes
      char* qbins = reinterpret_cast<char*>(mybins + qoff);
      auto bin = [&](int kk) -> float& { return *reinterpret_cast<float*>(qbins - knb[kk]); };
      if (fold) {
        float fa[kTile / 32][4], fb[kTile / 32][4];
#pragma unroll
        for (int kb = 0; kb < kTile / 32; ++kb)
#pragma unroll
          for (int g4 = 0; g4 < 4; ++g4) {
            const float d0 = dsb[kb][4 * g4], d1 = dsb[kb][4 * g4 + 1];
            const float d2 = dsb[kb][4 * g4 + 2], d3 = dsb[kb][4 * g4 + 3];
            float f = d3;
            f = d2 + fnext * dpp_lane<kDppNext>(f);
            f = d1 + fnext * dpp_lane<kDppNext>(f);
            fa[kb][g4] = d0 + fnext * dpp_lane<kDppNext>(f);
            const float p1 = dpp_lane<kDppWavePrev>(d2 * fsend);
            const float p2 = dpp_lane<kDppWavePrev>(dpp_lane<kDppWavePrev>(d1 * fsend) * fsend);
            fb[kb][g4] = fkeep * (d3 + p1 + p2);
          }
        // One update of this lane: the folded pair sums of key block kb,
        // group g4 (fa at (q, k), fb at (q, k+3)).
        auto upd = [&](int kb, int g4, float va, float vb) {
          const int kk = kb * 32 + 8 * g4 + 4 * half;
          if (va != 0.0f) bin(kk) += va;
          if (vb != 0.0f) bin(kk + 3) += vb;
        };
        if constexpr (kTile == 64) {
          // Both halves update with one instruction when their keys are at
          // least 32 tokens apart: the 32 queries of a half are consecutive
          // tokens, so (q, k) and (q', k') share a bin only if |k - k'| =
          // |q - q'| < 32.  Half 0 takes block 0 group t while half 1 takes
          // block 1 group t (keys 32 + 4 or more apart), then half 0 takes
          // block 1 group t while half 1 takes block 0 group t - 1 (36 or
          // more), and the two updates left over go alone.
          if (q0 + wave * kWaveQ + kWaveQ <= n && k0 + kTile <= n) {
            // Every query of the wave and every key of the tile is a window
            // token: the updates need no guard (adding 0 to a bin that no
            // other lane of the instruction touches changes nothing), and
            // the key words are read before the first update.  Word index of
            // this lane's group: 36 half + 8t in the first round, 32 - 36 half
            // + 8t in the second, 32 (half 0) or 28 (half 1) left over.
            float* w1[4][2];
            float* w2[3][2];
            float* wl[2];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const int kk = 36 * half + 8 * t;
              w1[t][0] = &bin(kk);
              w1[t][1] = &bin(kk + 3);
            }
#pragma unroll
            for (int t = 1; t < 4; ++t) {
              const int kk = 32 - 36 * half + 8 * t;
              w2[t - 1][0] = &bin(kk);
              w2[t - 1][1] = &bin(kk + 3);
            }
            {
              const int kk = half ? 28 : 32;
              wl[0] = &bin(kk);
              wl[1] = &bin(kk + 3);
            }
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              *w1[t][0] += half ? fa[1][t] : fa[0][t];
              *w1[t][1] += half ? fb[1][t] : fb[0][t];
            }
#pragma unroll
            for (int t = 1; t < 4; ++t) {
              *w2[t - 1][0] += half ? fa[0][t - 1] : fa[1][t];
              *w2[t - 1][1] += half ? fb[0][t - 1] : fb[1][t];
            }
            if (half == 0) { *wl[0] += fa[1][0]; *wl[1] += fb[1][0]; }
            __builtin_amdgcn_wave_barrier();
            if (half == 1) { *wl[0] += fa[0][3]; *wl[1] += fb[0][3]; }
            __builtin_amdgcn_wave_barrier();
          } else {
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const int kb = half, gt = t;
              upd(kb, gt, half ? fa[1][t] : fa[0][t], half ? fb[1][t] : fb[0][t]);
            }
#pragma unroll
            for (int t = 1; t < 4; ++t) {
              const int kb = 1 - half, gt = t - half;
              upd(kb, gt, half ? fa[0][t - 1] : fa[1][t], half ? fb[0][t - 1] : fb[1][t]);
            }
            if (half == 0) upd(1, 0, fa[1][0], fb[1][0]);
            __builtin_amdgcn_wave_barrier();
            if (half == 1) upd(0, 3, fa[0][3], fb[0][3]);
            __builtin_amdgcn_wave_barrier();
          }
        } else {
#pragma unroll 1
          for (int hh = 0; hh < 2; ++hh) {
            if (half == hh) {
#pragma unroll
              for (int g4 = 0; g4 < 4; ++g4) upd(0, g4, fa[0][g4], fb[0][g4]);
            }
            __builtin_amdgcn_wave_barrier();
          }
        }
        // pairs of runs shorter than three lanes that the fold left out
        if (__builtin_amdgcn_ballot_w64((run < 1 && rest < 2) || (run < 2 && rest < 1)) != 0) {
#pragma unroll 1
          for (int hh = 0; hh < 2; ++hh) {
            if (half == hh) {
#pragma unroll
              for (int kb = 0; kb < kTile / 32; ++kb)
#pragma unroll
                for (int g4 = 0; g4 < 4; ++g4) {
                  const int kk = kb * 32 + 8 * g4 + 4 * half;
#pragma unroll
                  for (int x = 1; x < 3; ++x)
                    if (run < x && rest < 3 - x && dsb[kb][4 * g4 + x] != 0.0f)
                      bin(kk + x) += dsb[kb][4 * g4 + x];
                }
            }
            __builtin_amdgcn_wave_barrier();
          }
        }
      } else {
#pragma unroll 1
        for (int hh = 0; hh < 2; ++hh) {
          if (half == hh) {
#pragma unroll
            for (int kb = 0; kb < kTile / 32; ++kb)
#pragma unroll
              for (int r = 0; r < 16; ++r) {
                if (dsb[kb][r] != 0.0f) bin(kb * 32 + acc_row(r, half)) += dsb[kb][r];
              }
          }
          __builtin_amdgcn_wave_barrier();
        }
      }
    }
    if (qvalid) {
      T* row = dq + wt.tok(g, qi) * g.C + hoff;
#pragma unroll
      for (int eb = 0; eb < HD / 32; ++eb)
#pragma unroll
        for (int grp = 0; grp < 4; ++grp) {
          const int e = eb * 32 + 8 * grp + 4 * half;
#pragma unroll
          for (int x = 0; x < 4; ++x) row[e + x] = from_float<T>(dqacc[eb][4 * grp + x] * scale);
        }
    }
  }
  lds_barrier();
  float* out = partial + ((int64_t)h * nslice + slice) * g.nbins;
  for (int x = threadIdx.x; x < g.nbins; x += kThreads)
    out[x] = ((dtab[x] + dtab[g.nbins + x]) + dtab[2 * g.nbins + x]) + dtab[3 * g.nbins + x];
}

// ---------------------------------------------------------------------------
// Backward, step 2: dK and dV.  Grid: B * nwin * heads * nkc (key chunks of
// 128; a wave owns 32 keys and walks the window's queries in LDS tiles).
// 16-bit types ask for two resident workgroups per CU: at head_dim 128 the
// compiler otherwise takes 280 registers (one wave per SIMD).  Capped at 256
// (two waves per SIMD) it keeps the matrix loop free of spills and spills 5
// (window-major) or 8 (NHWC) words of staging addresses, reloaded once per
// 64-query tile; the loop's lean form below took that down from 17 and 21
// words (backward -2 % at 1024-token windows, -6 % at 64-token ones).
// Three workgroups per CU (168 registers) spill inside the loop at
// head_dim 64 and run 25 % slower.
// ---------------------------------------------------------------------------
template <typename T, int HD, bool NHWC, bool QUAD>
__global__ __launch_bounds__(kThreads, sizeof(T) == 2 ? 2 : 1) void bwd_dkdv_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const T* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ D,
    const float* __restrict__ table, T* __restrict__ dk, T* __restrict__ dv,
    Geo g, int nkc, float scale_log2, float scale) {
  constexpr int kTile = tile_of<T, HD>();
  extern __shared__ __align__(16) char smem[];
  T* qr = reinterpret_cast<T*>(smem);                 // Q  [kTile][HD+kPad]
  T* dr = qr + kTile * (HD + kPad);                   // dO [kTile][HD+kPad]
  T* qtt = dr + kTile * (HD + kPad);                  // Q^T (transposed tile, fp32)
  T* dtt = qtt + ttile_size<T, HD>();                // dO^T (fp32)
  int* qinfo = reinterpret_cast<int*>(dtt + ttile_size<T, HD>());
  int* qnb = qinfo + kTile;                               // 4 x bias offset per query
  float* ql = reinterpret_cast<float*>(qnb + kTile);     // lse2 per query
  float* qd = ql + kTile;                                 // -D per query
  float* tab = qd + kTile;                                // [nbins+4], forward order
  uint32_t* tt = reinterpret_cast<uint32_t*>(tab + g.nbins + 4);   // [wh*ww] token offsets

  int bid = blockIdx.x;
  const int kc = bid % nkc; bid /= nkc;
  const int h = bid % g.heads; bid /= g.heads;
  const int w = bid % g.nwin;
  const int b = bid / g.nwin;
  const int i = w / g.Mw, j = w - (w / g.Mw) * g.Mw;
  const int cols = win_cols(g, j);
  const int n = win_rows(g, i) * cols;
  const int kbase = kc * kChunk;
  if (kbase >= n) return;
  const WinTokens<NHWC> wt(g, b, i, j);
  const int hoff = h * HD;
  const float bscale = sqrtf((float)HD);
  for (int x = threadIdx.x; x < g.nbins + 4; x += kThreads)
    tab[x] = x < g.nbins ? table[x * g.heads + h] * bscale : -INFINITY;
  const bool mask = window_has_labels(g, i, j) || (n % kTile) != 0;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int ki = kbase + wave * kWaveQ + col;
  const bool kvalid = ki < n;
  const bool wactive = kbase + wave * kWaveQ < n;   // else staging and barriers only
  const int kinf = token_info(g, i, j, cols, kvalid ? ki : 0, n);
  const int klab = kvalid ? (kinf >> 24) : 0xFE;
  const int kfwd = (g.wh - 1) * g.bstride + (g.ww - 1) - (kinf & 0xFFFFFF);
  const char* tabk = reinterpret_cast<const char*>(tab + kfwd);
  const float inv_sl2 = 1.0f / scale_log2;

  typename Operand<T>::type kop[HD / 16], vop[HD / 16];
#pragma unroll
  for (int c = 0; c < HD / 16; ++c) {
    kop[c] = kvalid ? load_op_global<T>(k + wt.tok(g, ki) * g.C + hoff + 16 * c + 8 * half)
                    : zero_op<T>();
    vop[c] = kvalid ? load_op_global<T>(v + wt.tok(g, ki) * g.C + hoff + 16 * c + 8 * half)
                    : zero_op<T>();
  }
  f32x16 dkacc[HD / 32], dvacc[HD / 32];
#pragma unroll
  for (int eb = 0; eb < HD / 32; ++eb) { dkacc[eb] = f32x16{}; dvacc[eb] = f32x16{}; }

  // Q, dO tiles go HBM -> registers -> LDS, one tile ahead up to head dim 64
  constexpr bool kPrefetch = HD <= 64;
  TileRegs<T, HD> rq, rd;
  if (kPrefetch) {
    tile_load(rq, q, g, wt, 0, n, hoff);
    tile_load(rd, dout, g, wt, 0, n, hoff);
  }
  // Head dim 128 (no register prefetch of the tiles): the rows come from
  // the token table, and the per-query words of the next tile are loaded
  // right after the staging barrier so that no wave waits at the barrier for
  // their global loads (backward -7 % at 1024-token windows).  Up to head
  // dim 64 the plain form measured 2 % faster.
  constexpr bool kTab = !kPrefetch;
  if constexpr (kTab) {
    tok_fill(tt, g, wt, n);
    if (NHWC) lds_barrier();   // the first tile comes from the table too
  }
  // Per-query words of a tile (threads below kTile): label/bias word,
  // log-sum-exp in log2 units (+inf for padding queries: P = 0) and -D (the
  // dP accumulator's start).
  int winf = 0;
  float wl = INFINITY, wd = 0.0f;
  auto words = [&](int t0) {
    if (threadIdx.x < kTile) {
      const int t = t0 + threadIdx.x;
      winf = token_info(g, i, j, cols, t, n);
      const int64_t li = t < n ? wt.lse_at(g, h, t) : 0;
      wl = t < n ? lse[li] * kLog2e : INFINITY;
      wd = t < n ? -D[li] : 0.0f;
    }
  };
  if constexpr (kTab) words(0);
  for (int t0 = 0; t0 < n; t0 += kTile) {
    if constexpr (kTab) {
      tile_load_tt(rq, q, g, wt, tt, t0, n, hoff);
      tile_load_tt(rd, dout, g, wt, tt, t0, n, hoff);
    }
    lds_barrier();
    tile_store<T, HD, true, sizeof(T) == 4>(rq, qr, qtt);
    tile_store<T, HD, true, sizeof(T) == 4>(rd, dr, dtt);
    if (threadIdx.x < kTile) {
      if constexpr (kTab) {
        qinfo[threadIdx.x] = winf;
        qnb[threadIdx.x] = 4 * (winf & 0xFFFFFF);
        ql[threadIdx.x] = wl;
        qd[threadIdx.x] = wd;
      } else {
        const int t = t0 + threadIdx.x;
        const int inf = token_info(g, i, j, cols, t, n);
        qinfo[threadIdx.x] = inf;
        qnb[threadIdx.x] = 4 * (inf & 0xFFFFFF);
        const int64_t li = t < n ? wt.lse_at(g, h, t) : 0;
        ql[threadIdx.x] = t < n ? lse[li] * kLog2e : INFINITY;
        qd[threadIdx.x] = t < n ? -D[li] : 0.0f;
      }
    }
    lds_barrier();
    if (t0 + kTile < n) {
      if constexpr (kTab) {
        words(t0 + kTile);
      } else {
        tile_load(rq, q, g, wt, t0 + kTile, n, hoff);
        tile_load(rd, dout, g, wt, t0 + kTile, n, hoff);
      }
    }
    if (!wactive) continue;
    // head_dim 128: one 32-query block at a time (unrolled, the two blocks'
    // operands overlap and the 256 registers spill)
#pragma unroll(HD == 128 ? 1 : kTile / 32)
    for (int qb = 0; qb < kTile / 32; ++qb) {
      // registers 4g..4g+3 hold queries 32qb + 8g + 4*half + 0..3: their
      // log-sum-exp and D are four consecutive LDS words.
      // At head_dim 128 the score accumulator starts at bias - LSE (in
      // score units), as the dP one starts at -D, so that no per-query value
      // stays in registers across the products, and dS replaces dP in place
      // (-20 % spill there; at head_dim 64 the plain form is 1.5 % faster).
      constexpr bool kLean = HD == 128;
      // up to head dim 64, the block's Q and dO operands are read from LDS
      // before its bias (-1 % at 576-token windows)
      constexpr bool kHold = HD <= 64;
      typename Operand<T>::type qo_[kHold ? HD / 16 : 1], do_[kHold ? HD / 16 : 1];
      if constexpr (kHold) {
#pragma unroll
        for (int c = 0; c < HD / 16; ++c) {
          qo_[c] = load_op_lds<T>(qr + (qb * 32 + col) * (HD + kPad) + 16 * c + 8 * half);
          do_[c] = load_op_lds<T>(dr + (qb * 32 + col) * (HD + kPad) + 16 * c + 8 * half);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      // (the byte-offset form costs head dim 128 extra spill)
      f32x16 s;
      if constexpr (HD <= 64)
        s = mask ? bias_init_t_nb<QUAD, true>(qinfo, qnb, tabk, qb, half, klab)
                 : bias_init_t_nb<QUAD, false>(qinfo, qnb, tabk, qb, half, klab);
      else
        s = mask ? bias_init_t<QUAD, true>(qinfo, tab, qb, half, kfwd, klab, g.nbins)
                 : bias_init_t<QUAD, false>(qinfo, tab, qb, half, kfwd, klab, g.nbins);
      f32x16 dp, lq;
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const f32x4 d4 = *reinterpret_cast<const f32x4*>(qd + qb * 32 + 8 * g4 + 4 * half);
        const f32x4 l4 = *reinterpret_cast<const f32x4*>(ql + qb * 32 + 8 * g4 + 4 * half);
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          dp[4 * g4 + x] = d4[x];      // dP - D straight from the product
          if constexpr (kLean) s[4 * g4 + x] -= l4[x] * inv_sl2;
          else lq[4 * g4 + x] = l4[x];
        }
      }
#pragma unroll
      for (int c = 0; c < HD / 16; ++c) {
        if constexpr (kHold) {
          mma16(s, qo_[c], kop[c]);
          mma16(dp, do_[c], vop[c]);
        } else {
          mma16(s, load_op_lds<T>(qr + (qb * 32 + col) * (HD + kPad) + 16 * c + 8 * half), kop[c]);
          mma16(dp, load_op_lds<T>(dr + (qb * 32 + col) * (HD + kPad) + 16 * c + 8 * half), vop[c]);
        }
      }
      f32x16 dsr;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = kLean ? __builtin_amdgcn_exp2f(s[r] * scale_log2)
                              : __builtin_amdgcn_exp2f(s[r] * scale_log2 - lq[r]);
        if constexpr (kLean) dp[r] *= p;          // dS
        else dsr[r] = p * dp[r];
        s[r] = p;
      }
      const f32x16& ds = kLean ? dp : dsr;
#pragma unroll
      for (int eb = 0; eb < HD / 32; ++eb) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          if constexpr (sizeof(T) == 2) {
            mma16(dvacc[eb], lds_tr_op<T, HD + kPad>(dr, qb, c, eb, lane), pack8<T>(s, 8 * c));
            mma16(dkacc[eb], lds_tr_op<T, HD + kPad>(qr, qb, c, eb, lane), pack8<T>(ds, 8 * c));
          } else {
            const int cofs = qb * 32 + 16 * c;
            mma16(dvacc[eb], load_op_lds_perm<T>(dtt + tr_row<T, HD>(eb * 32 + col) + cofs, half),
                  pack8<T>(s, 8 * c));
            mma16(dkacc[eb], load_op_lds_perm<T>(qtt + tr_row<T, HD>(eb * 32 + col) + cofs, half),
                  pack8<T>(ds, 8 * c));
          }
        }
      }
    }
  }
  if (!kvalid) return;
  T* krow = dk + wt.tok(g, ki) * g.C + hoff;
  T* vrow = dv + wt.tok(g, ki) * g.C + hoff;
#pragma unroll
  for (int eb = 0; eb < HD / 32; ++eb)
#pragma unroll
    for (int grp = 0; grp < 4; ++grp) {
      const int e = eb * 32 + 8 * grp + 4 * half;
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        krow[e + x] = from_float<T>(dkacc[eb][4 * grp + x] * scale);
        vrow[e + x] = from_float<T>(dvacc[eb][4 * grp + x]);
      }
    }
}

// ---------------------------------------------------------------------------
// Host-side launchers (called by the C ABI after validation).
// ---------------------------------------------------------------------------
static inline int num_chunks(const Geo& g) { return (g.wh * g.ww + kChunk - 1) / kChunk; }


template <typename T, int HD>
static size_t fwd_lds(const Geo& g) {
  constexpr int kTile = tile_of<T, HD>();
  return sizeof(T) * (kTile * (HD + kPad) + vtile_size<T, HD>()) + 4 * kTile + 4 * (g.nbins + 4) +
         4 * g.wh * g.ww;
}
// Key tiles the dQ kernel keeps resident for a whole item: every tile of the
// window for 16-bit types, head_dim up to 64 and windows of up to 256 tokens
// (the staging then happens once per item instead of once per tile and
// sweep), else 1 (tiles streamed through one staging buffer).
template <typename T, int HD>
static int dq_tiles(const Geo& g) {
  constexpr int kTile = tile_of<T, HD>();
  if (sizeof(T) != 2 || HD > 64 || g.wh * g.ww > 256) return 1;
  return (g.wh * g.ww + kTile - 1) / kTile;
}
template <typename T, int HD>
static size_t dq_lds(const Geo& g) {
  constexpr int kTile = tile_of<T, HD>();
  const int nt = dq_tiles<T, HD>(g);
  return sizeof(T) * (2 * nt * kTile * (HD + kPad) + ttile_size<T, HD>()) + 8 * nt * kTile +
         4 * (g.nbins + 4) + 16 * g.nbins + 4 * g.wh * g.ww;
}
template <typename T, int HD>
static size_t dkdv_lds(const Geo& g) {
  constexpr int kTile = tile_of<T, HD>();
  return sizeof(T) * (2 * kTile * (HD + kPad) + 2 * ttile_size<T, HD>()) + 16 * kTile + 4 * (g.nbins + 4) +
         (HD > 64 ? 4 * g.wh * g.ww : 0);    // token table (head dim 128 only)
}

// Per-head slices of the dQ / bias-gradient kernel.  The grid is one round
// of resident workgroups rounded down to whole heads: a grid a few
// workgroups past a round leaves those few to run alone at the end (24 heads
// with ceil(2048 / 24) slices each made 2064 workgroups, 4 rounds and 16
// more).  Measured against 2, 4 and 8 rounds, one was fastest or level on
// every workload.  The launcher asks the runtime how many workgroups one CU
// holds; the workspace (a pure function of the geometry and element type, so
// that it can be queried) is sized for the most the kernel's LDS allows.
constexpr int kF32 = 0, kBF16 = 1;
static int slices_for(const Geo& g, int per_cu) {
  const int items = g.B * g.nwin * num_chunks(g);
  int n = g.cus * per_cu / g.heads;
  if (n > items) n = items;
  return n < 1 ? 1 : n;
}
template <typename T>
static int bwd_nslice_max_t(const Geo& g) {
  const size_t lds = g.hd == 32 ? dq_lds<T, 32>(g) : g.hd == 64 ? dq_lds<T, 64>(g) : dq_lds<T, 128>(g);
  int per_cu = (int)((160 * 1024) / lds);            // four waves a workgroup, at most 32 a CU
  if (per_cu > 8) per_cu = 8;
  return slices_for(g, per_cu < 1 ? 1 : per_cu);
}
int bwd_nslice(const Geo& g, int dt) {
  return dt == kF32 ? bwd_nslice_max_t<float>(g) : dt == kBF16 ? bwd_nslice_max_t<__bf16>(g)
                                                               : bwd_nslice_max_t<_Float16>(g);
}

template <typename T, int HD, bool NHWC>
static hipError_t fwd_impl(const Geo& g, const void* q, const void* k, const void* v,
                           const float* table, void* o, void* olo, float* lse, hipStream_t st) {
  const int nqc = num_chunks(g);
  const int grid = grid8(g.B * g.nwin * g.heads * nqc);
  const float sl2 = kLog2e / sqrtf((float)HD);
  const size_t lds = fwd_lds<T, HD>(g);
#define TERRA_LAUNCH_FWD(QD, SP)                                                                  \
  hipLaunchKernelGGL((fwd_kernel<T, HD, NHWC, QD, SP>), dim3(grid), dim3(kThreads), lds, st,       \
                     (const T*)q, (const T*)k, (const T*)v, table, (T*)o, (T*)olo, lse, g, nqc, sl2)
  const bool quad = quad_layout(g);
  if constexpr (sizeof(T) == 2) {
    if (olo != nullptr) {
      if (quad) TERRA_LAUNCH_FWD(true, true);
      else TERRA_LAUNCH_FWD(false, true);
      return hipGetLastError();
    }
  }
  if (quad) TERRA_LAUNCH_FWD(true, false);
  else TERRA_LAUNCH_FWD(false, false);
#undef TERRA_LAUNCH_FWD
  return hipGetLastError();
}

size_t bwd_workspace(const Geo& g, int dt) {
  if (win_bwd_ok(g, dt == 1)) return (size_t)g.heads * win_bwd_nslice(g) * g.nbins * sizeof(float);
  const size_t dbytes = (size_t)g.B * g.heads * g.HW * sizeof(float);
  const size_t pbytes = (size_t)g.heads * bwd_nslice(g, dt) * g.nbins * sizeof(float);
  return ((dbytes + 255) / 256) * 256 + pbytes;
}

template <typename T, int HD, bool NHWC>
static hipError_t bwd_impl(const Geo& g, const void* q, const void* k, const void* v,
                           const void* o, const void* olo, const void* dout, const float* lse,
                           const float* table, void* dq, void* dk, void* dv, float* dtab,
                           void* ws, hipStream_t st) {
  const size_t dbytes = (size_t)g.B * g.heads * g.HW * sizeof(float);
  float* D = reinterpret_cast<float*>(ws);
  float* partial = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + ((dbytes + 255) / 256) * 256);
  hipError_t e;
  const int nqc = num_chunks(g);
  const float sl2 = kLog2e / sqrtf((float)HD);
  const float scale = 1.0f / sqrtf((float)HD);
  const size_t lds_dq = dq_lds<T, HD>(g);
  const bool quad = quad_layout(g);
  const bool res = dq_tiles<T, HD>(g) > 1;
  const void* dq_fn;
  if constexpr (sizeof(T) == 2 && HD <= 64) {
    dq_fn = quad ? (res ? reinterpret_cast<const void*>(&bwd_dq_kernel<T, HD, NHWC, true, true>)
                        : reinterpret_cast<const void*>(&bwd_dq_kernel<T, HD, NHWC, true, false>))
                 : (res ? reinterpret_cast<const void*>(&bwd_dq_kernel<T, HD, NHWC, false, true>)
                        : reinterpret_cast<const void*>(&bwd_dq_kernel<T, HD, NHWC, false, false>));
  } else {
    dq_fn = quad ? reinterpret_cast<const void*>(&bwd_dq_kernel<T, HD, NHWC, true, false>)
                 : reinterpret_cast<const void*>(&bwd_dq_kernel<T, HD, NHWC, false, false>);
  }
  int resident = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&resident, dq_fn, kThreads, lds_dq) != hipSuccess) {
    (void)hipGetLastError();
    resident = 2;
  }
  int nslice = slices_for(g, resident < 1 ? 1 : resident);
  const int nmax = bwd_nslice_max_t<T>(g);
  if (nslice > nmax) nslice = nmax;
#define TERRA_LAUNCH_DQ(QD, RS)                                                                 \
  hipLaunchKernelGGL((bwd_dq_kernel<T, HD, NHWC, QD, RS>), dim3(g.heads * nslice), dim3(kThreads),  \
                     lds_dq, st, (const T*)q, (const T*)k, (const T*)v, (const T*)o, (const T*)olo,  \
                     (const T*)dout, lse, D, table, (T*)dq, partial, g, nqc, nslice, sl2, scale)
  if constexpr (sizeof(T) == 2 && HD <= 64) {
    if (quad && res) TERRA_LAUNCH_DQ(true, true);
    else if (quad) TERRA_LAUNCH_DQ(true, false);
    else if (res) TERRA_LAUNCH_DQ(false, true);
    else TERRA_LAUNCH_DQ(false, false);
  } else {
    if (quad) TERRA_LAUNCH_DQ(true, false);
    else TERRA_LAUNCH_DQ(false, false);
  }
#undef TERRA_LAUNCH_DQ
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int grid = g.B * g.nwin * g.heads * nqc;
  const size_t lds_kv = dkdv_lds<T, HD>(g);
  if (quad)
    hipLaunchKernelGGL((bwd_dkdv_kernel<T, HD, NHWC, true>), dim3(grid), dim3(kThreads), lds_kv, st,
                       (const T*)q, (const T*)k, (const T*)v, (const T*)dout, lse, D, table,
                       (T*)dk, (T*)dv, g, nqc, sl2, scale);
  else
    hipLaunchKernelGGL((bwd_dkdv_kernel<T, HD, NHWC, false>), dim3(grid), dim3(kThreads), lds_kv, st,
                       (const T*)q, (const T*)k, (const T*)v, (const T*)dout, lse, D, table,
                       (T*)dk, (T*)dv, g, nqc, sl2, scale);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_dtab_reduce(g, partial, dtab, nslice, st);
}

// Element type codes of the C ABI: 0 float, 1 bfloat16, 2 float16.

template <typename T>
static size_t max_lds_t(const Geo& g) {
  size_t m, d;
  switch (g.hd) {
    case 32: m = dkdv_lds<T, 32>(g); d = dq_lds<T, 32>(g); break;
    case 64: m = dkdv_lds<T, 64>(g); d = dq_lds<T, 64>(g); break;
    default: m = dkdv_lds<T, 128>(g); d = dq_lds<T, 128>(g); break;
  }
  return m > d ? m : d;
}

size_t attn_max_lds(const Geo& g, int dt) {
  size_t m = dt == kF32 ? max_lds_t<float>(g) : dt == kBF16 ? max_lds_t<__bf16>(g) : max_lds_t<_Float16>(g);
  const bool bf = dt == kBF16;
  if (win_fwd_ok(g, bf) && win_fwd_lds(g) > m) m = win_fwd_lds(g);
  if (win_bwd_ok(g, bf) && win_bwd_lds(g) > m) m = win_bwd_lds(g);
  return m;
}

template <typename T, bool NHWC>
static hipError_t fwd_generic(const Geo& g, const void* q, const void* k, const void* v,
                              const float* table, void* o, void* olo, float* lse, hipStream_t st) {
  switch (g.hd) {
    case 32: return fwd_impl<T, 32, NHWC>(g, q, k, v, table, o, olo, lse, st);
    case 64: return fwd_impl<T, 64, NHWC>(g, q, k, v, table, o, olo, lse, st);
    default: return fwd_impl<T, 128, NHWC>(g, q, k, v, table, o, olo, lse, st);
  }
}

template <typename T, bool NHWC>
static hipError_t bwd_generic(const Geo& g, const void* q, const void* k, const void* v,
                              const void* o, const void* olo, const void* dout, const float* lse,
                              const float* table, void* dq, void* dk, void* dv, float* dtab, void* ws,
                              hipStream_t st) {
  switch (g.hd) {
    case 32: return bwd_impl<T, 32, NHWC>(g, q, k, v, o, olo, dout, lse, table, dq, dk, dv, dtab, ws, st);
    case 64: return bwd_impl<T, 64, NHWC>(g, q, k, v, o, olo, dout, lse, table, dq, dk, dv, dtab, ws, st);
    default: return bwd_impl<T, 128, NHWC>(g, q, k, v, o, olo, dout, lse, table, dq, dk, dv, dtab, ws, st);
  }
}

template <bool NHWC>
static hipError_t fwd_dispatch(const Geo& g, int dt, const void* q, const void* k, const void* v,
                               const float* table, void* o, void* olo, float* lse, hipStream_t st) {
  if (dt == kF32) return fwd_generic<float, NHWC>(g, q, k, v, table, o, nullptr, lse, st);
  if (dt == kBF16) return fwd_generic<__bf16, NHWC>(g, q, k, v, table, o, olo, lse, st);
  return fwd_generic<_Float16, NHWC>(g, q, k, v, table, o, olo, lse, st);
}

template <bool NHWC>
static hipError_t bwd_dispatch(const Geo& g, int dt, const void* q, const void* k, const void* v,
                               const void* o, const void* olo, const void* dout, const float* lse,
                               const float* table, void* dq, void* dk, void* dv, float* dtab, void* ws,
                               hipStream_t st) {
  if (dt == kF32)
    return bwd_generic<float, NHWC>(g, q, k, v, o, nullptr, dout, lse, table, dq, dk, dv, dtab, ws, st);
  if (dt == kBF16)
    return bwd_generic<__bf16, NHWC>(g, q, k, v, o, olo, dout, lse, table, dq, dk, dv, dtab, ws, st);
  return bwd_generic<_Float16, NHWC>(g, q, k, v, o, olo, dout, lse, table, dq, dk, dv, dtab, ws, st);
}

// True when the forward writes the rounding residual O_lo and the backward
// takes D from it: 16-bit types on the generic kernels with windows of more
// than 256 tokens.  Smaller windows keep the D sweep, which is cheaper there
// than the split P V product plus the O_lo traffic (measured: 144-token
// windows, hd 32: forward +0.017 ms, backward -0.011 ms; 64-token windows,
// hd 128: forward +0.10 ms, backward +0.10 ms; 576-token windows, hd 64:
// forward +0.26 ms, backward -0.81 ms).
bool attn_uses_olo(const Geo& g, int dt) {
  return dt != kF32 && !win_fwd_ok(g, dt == kBF16) && !win_bwd_ok(g, dt == kBF16) && g.wh * g.ww > 256;
}

// dt: element type code.  nhwc: q, k, v, o (and dout, dq, dk, dv) are
// B x H x W x C read and written in place (the token route fused into the
// kernels), LSE in the same token order; otherwise they are window-major.
// olo (nullable) is written and read only where attn_uses_olo holds.
hipError_t launch_attn_fwd(const Geo& g, int dt, bool nhwc, const void* q, const void* k,
                           const void* v, const float* table, void* o, void* olo, float* lse,
                           hipStream_t st) {
  if (win_fwd_ok(g, dt == kBF16)) return launch_win_fwd(g, nhwc, q, k, v, table, o, lse, st);
  if (!attn_uses_olo(g, dt)) olo = nullptr;
  return nhwc ? fwd_dispatch<true>(g, dt, q, k, v, table, o, olo, lse, st)
              : fwd_dispatch<false>(g, dt, q, k, v, table, o, olo, lse, st);
}

hipError_t launch_attn_bwd(const Geo& g, int dt, bool nhwc, const void* q, const void* k,
                           const void* v, const void* o, const void* olo, const void* dout,
                           const float* lse, const float* table, void* dq, void* dk, void* dv,
                           float* dtab, void* ws, hipStream_t st) {
  if (win_bwd_ok(g, dt == kBF16)) {
    const int nslice = win_bwd_nslice(g);
    float* partial = reinterpret_cast<float*>(ws);
    hipError_t e = launch_win_bwd(g, nhwc, q, k, v, dout, lse, table, dq, dk, dv, partial, nslice, st);
    if (e != hipSuccess) return e;
    return launch_dtab_reduce(g, partial, dtab, nslice, st);
  }
  if (!attn_uses_olo(g, dt)) olo = nullptr;
  return nhwc ? bwd_dispatch<true>(g, dt, q, k, v, o, olo, dout, lse, table, dq, dk, dv, dtab, ws, st)
              : bwd_dispatch<false>(g, dt, q, k, v, o, olo, dout, lse, table, dq, dk, dv, dtab, ws, st);
}

}  // namespace terra
