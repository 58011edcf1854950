// terra_common.h - device-side helpers shared by the gfx950 kernels.
//
// Window geometry in closed form (Sec. IV-D, Eq. (2) generalised to a
// wh x ww window, ragged last row/column, row-major window order of
// Sec. V-A), the packed kernel argument block, and thin wrappers around the
// CDNA4 matrix-core instructions used by the attention kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace terra {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Everything a kernel needs to know about the grid, passed by value.
struct Geo {
  int B, H, W, C, heads, hd;
  int wh, ww, sh, sw, flags;
  int Mh, Mw, nwin;   // window grid; nwin = Mh * Mw per image
  int HW;
  int nbins;          // (2wh-1)(2ww-1)
  int bstride;        // 2ww-1
  // Row stride and size of the window kernels' LDS bias table: rows padded
  // to a stride of 16 mod 32 so that the table reads of two window rows of
  // queries fall in distinct LDS banks.
  int tstride, ntab;  // ntab = (2wh-1) * tstride
  // 1 / width of full-width windows and of the last column's windows (the
  // float reciprocals fast_div starts from), set on the host.
  float rcols[2];
  // Compute units the persistent grids are sized for: the device's count at
  // launch; kMaxCus when sizing workspaces, which are pure functions of the
  // geometry (every slice count grows with it, so a workspace sized for
  // kMaxCus covers any device up to that many).
  int cus;
};

constexpr int kMaxCus = 512;

__host__ inline void set_table_stride(Geo& g) {
  g.tstride = g.bstride + ((48 - g.bstride % 32) % 32);
  g.ntab = (2 * g.wh - 1) * g.tstride;
}

// Extent of window row i / column j (partial at the far edge).
__device__ __host__ inline int win_rows(const Geo& g, int i) {
  int r = g.H - i * g.wh;
  return r < g.wh ? r : g.wh;
}
__device__ __host__ inline int win_cols(const Geo& g, int j) {
  int c = g.W - j * g.ww;
  return c < g.ww ? c : g.ww;
}

__host__ inline void set_col_recips(Geo& g) {
  g.rcols[0] = 1.0f / (float)win_cols(g, 0);
  g.rcols[1] = 1.0f / (float)win_cols(g, g.Mw - 1);
}

// Sum and maximum over the two 32-lane halves of a wave, in every lane:
// swapping the upper half of x with the lower half of a copy of x leaves
// the lower half's value in one and the upper half's in the other.  Written
// as assembly (with wait states around it) because the compiler folds the
// two results of the built-in swap of equal operands into one.
__device__ __forceinline__ float2 halves_pair(float x) {
  float y = x;
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(x), "+v"(y));
  return float2{x, y};
}
__device__ __forceinline__ float halves_sum(float x) {
  const float2 p = halves_pair(x);
  return p.x + p.y;
}
__device__ __forceinline__ float halves_max(float x) {
  const float2 p = halves_pair(x);
  return fmaxf(p.x, p.y);
}

// Reciprocal of the width of window column j.
__device__ inline float win_rcols(const Geo& g, int j) { return j == g.Mw - 1 ? g.rcols[1] : g.rcols[0]; }
// First window-major slot of window (i, j) within its image: all window rows
// above i are full (wh rows each), and the windows to the left in row i hold
// rows_i * ww tokens each.
__device__ __host__ inline int win_offset(const Geo& g, int i, int j) {
  return i * g.wh * g.W + win_rows(g, i) * j * g.ww;
}
// Wrap labels of rolled row r / rolled column s (bit 0 latitude, bit 1 longitude).
__device__ __host__ inline int row_label(const Geo& g, int r) {
  return ((g.flags & 1) && g.sh > 0 && r >= g.H - g.sh) ? 1 : 0;
}
__device__ __host__ inline int col_label(const Geo& g, int s) {
  return ((g.flags & 2) && g.sw > 0 && s >= g.W - g.sw) ? 2 : 0;
}

// n / d for 0 <= n < 2^22, 1 <= d < 2^16, via a float reciprocal and one
// correction step each way.
__device__ inline int fast_div(int n, int d, float rcp) {
  int q = (int)((float)n * rcp);
  int r = n - q * d;
  if (r < 0) { q -= 1; }
  else if (r >= d) { q += 1; }
  return q;
}

// Token index of row t of window (b, i, j) in a B x H x W x C tensor read in
// one of two layouts:
// * window-major (routed): the window's first slot plus t;
// * NHWC, in place: the grid point that the rolled coordinate
//   (i*wh + a, j*ww + c), (a, c) = (t / cols, t % cols), was taken from,
//   ((i*wh + a + sh) mod H, (j*ww + c + sw) mod W) - the cyclic shift of
//   Sec. IV-D read as a roll by -shift, so reading in place fuses the token
//   route (and writing in place its inverse) into the attention kernels.
// The log-sum-exp (and the backward's D) of a token sits at
// (b*heads + h)*HW + (token - b*HW) in either layout.
template <bool NHWC>
struct WinTokens {
  // Attention tensors hold fewer than 2^31 elements, so token indices and
  // element offsets fit 32 bits.
  uint32_t img0, first;   // b*HW; window-major first slot of the window
  int r0, c0, cols;       // i*wh + sh, j*ww + sw, window width
  float rcols;
  __device__ WinTokens(const Geo& g, int b, int i, int j)
      : img0((uint32_t)(b * g.HW)), first((uint32_t)(b * g.HW + win_offset(g, i, j))),
        r0(i * g.wh + g.sh), c0(j * g.ww + g.sw), cols(win_cols(g, j)), rcols(win_rcols(g, j)) {}
  // Both wraps subtract once: the rolled coordinate is below twice the
  // extent, and for x < 2 L, min(x, x - L) over unsigned is x mod L.
  __device__ uint32_t tok(const Geo& g, int t) const {
    if (!NHWC) return first + t;
    const int a = fast_div(t, cols, rcols);
    uint32_t u = (uint32_t)(r0 + a);
    u = min(u, u - (uint32_t)g.H);
    uint32_t v = (uint32_t)(c0 + (t - a * cols));
    v = min(v, v - (uint32_t)g.W);
    return img0 + u * (uint32_t)g.W + v;
  }
  __device__ uint32_t lse_at(const Geo& g, int h, int t) const {
    return img0 * (uint32_t)g.heads + (uint32_t)(h * g.HW) + (tok(g, t) - img0);
  }
};

// True when window (wi, wj) holds tokens of more than one wrap label (the
// latitude rows or longitude columns that the shift moved across the edge).
__device__ inline bool window_has_labels(const Geo& g, int wi, int wj) {
  const bool lat = (g.flags & 1) && g.sh > 0 && (wi * g.wh + win_rows(g, wi)) > g.H - g.sh;
  const bool lon = (g.flags & 2) && g.sw > 0 && (wj * g.ww + win_cols(g, wj)) > g.W - g.sw;
  return lat || lon;
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

// The same in the key-major form (lane = key, registers = queries of query
// block QB): the table is in forward bin order, times sqrt(hd), with four
// -inf entries after it; kfwd is the lane's key term of the bin index,
// (wh-1)(2ww-1) + ww-1 - (a_k (2ww-1) + c_k), and klab its label.
template <bool QUAD, bool MASK>
__device__ inline f32x16 bias_init_t(const int* qinfo, const float* tabf, int qb, int half, int kfwd,
                                     int klab, int nbins) {
  f32x16 c;
#pragma unroll
  for (int g4 = 0; g4 < 4; ++g4) {
    int inf = qinfo[32 * qb + 8 * g4 + 4 * half];
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      if (!QUAD && x > 0) inf = qinfo[32 * qb + 8 * g4 + 4 * half + x];
      int rb = kfwd + (inf & 0xFFFFFF);
      if (MASK && (inf >> 24) != klab) rb = nbins - (QUAD ? x : 0);
      c[4 * g4 + x] = tabf[rb + (QUAD ? x : 0)];
    }
  }
  return c;
}

// Four consecutive result registers are four consecutive keys (queries) of
// one window row, with one label, when every window width is a multiple of
// 4 and the longitude wrap is not masked.
__host__ inline bool quad_layout(const Geo& g) {
  return g.ww % 4 == 0 && (g.W % g.ww) % 4 == 0 && (g.flags & 2) == 0;
}

// Value of another lane by a DPP move (0 where the source lane is absent).
template <int CTRL>
__device__ __forceinline__ float dpp_lane(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, true));
}
constexpr int kDppNext = 0x130;    // wave_shl:1 - lane l reads lane l+1
constexpr int kDppPrev1 = 0x111;   // row_shr:1  - lane l reads lane l-1 (same 16-lane row)
constexpr int kDppPrev2 = 0x112;   // row_shr:2  - lane l reads lane l-2
constexpr int kDppWavePrev = 0x138;  // wave_shr:1 - lane l reads lane l-1

// ---------------------------------------------------------------------------
// Matrix-core tiles.  One MFMA "operand" is 8 consecutive contraction-dim
// elements per lane: lane l supplies row/column (l % 32) and contraction
// slots 8*(l/32) .. 8*(l/32)+7 of a 16-deep chunk.  The 32x32 float result
// D[m][n] sits in lane n + 32*((m/4)%2), register (m%4) + 4*(m/8).
// ---------------------------------------------------------------------------
template <typename T> struct Operand;
template <> struct Operand<__bf16> { typedef bf16x8 type; };
template <> struct Operand<_Float16> { typedef f16x8 type; };
template <> struct Operand<float> { typedef f32x8 type; };

// Transposed operand of channel block eb, key block kb, chunk c2 from a
// row-major 16-bit tile V in LDS of row stride VS (elements): lane
// (channel col, half) receives V[32 kb + 16 c2 + 4 half + x][32 eb + col]
// and the same 8 rows further, x = 0..3 (two runs of 4 keys, the slot order
// of the 32x32 result registers).  In each 16-lane group G of the LDS
// transpose read, lane i receives element i % 4 of the 8 bytes addressed by
// lane 16 G + 4 x + i / 4, x = 0..3; so lane L addresses row
// 32 kb + 16 c2 + 4 (G / 2) + (L / 4) % 4, channels 32 eb + 16 (G % 2) + 4 (L % 4).
template <typename T, int VS>
__device__ inline typename Operand<T>::type lds_tr_op(const T* V, int kb, int c2, int eb, int lane) {
  typedef short v4s __attribute__((ext_vector_type(4)));
  typedef short v8s __attribute__((ext_vector_type(8)));
  typedef __attribute__((address_space(3))) v4s lds_v4s;
  const int G = lane >> 4, x = (lane >> 2) & 3, m = lane & 3;
  const T* p = V + (32 * kb + 16 * c2 + 4 * (G >> 1) + x) * VS + 32 * eb + 16 * (G & 1) + 4 * m;
  const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)p);
  const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(p + 8 * VS));
  const v8s o = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(typename Operand<T>::type, o);
}

__device__ inline void mma16(f32x16& acc, const bf16x8& a, const bf16x8& b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
}
__device__ inline void mma16(f32x16& acc, const f16x8& a, const f16x8& b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc, 0, 0, 0);
}
// fp32: eight 32x32x2 steps; step i contracts slot i of both lane halves, so
// the slot numbering matches the bf16 instruction exactly.
__device__ inline void mma16(f32x16& acc, const f32x8& a, const f32x8& b) {
#pragma unroll
  for (int i = 0; i < 8; ++i)
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[i], acc, 0, 0, 0);
}

// Result-register index -> row m within the 32x32 tile, for lane half h.
__device__ __host__ constexpr int acc_row(int r, int h) { return 8 * (r / 4) + 4 * h + (r % 4); }

template <typename T> __device__ inline T from_float(float x);
template <> __device__ inline float from_float<float>(float x) { return x; }
template <> __device__ inline __bf16 from_float<__bf16>(float x) { return (__bf16)x; }
template <> __device__ inline _Float16 from_float<_Float16>(float x) { return (_Float16)x; }

template <typename T> __device__ inline float to_float(T x);
template <> __device__ inline float to_float<float>(float x) { return x; }
template <> __device__ inline float to_float<__bf16>(__bf16 x) { return (float)x; }
template <> __device__ inline float to_float<_Float16>(_Float16 x) { return (float)x; }

// Pack result registers r0..r0+7 (as float) into an operand.
template <typename T>
__device__ inline typename Operand<T>::type pack8(const f32x16& acc, int r0) {
  typename Operand<T>::type o;
#pragma unroll
  for (int i = 0; i < 8; ++i) o[i] = from_float<T>(acc[r0 + i]);
  return o;
}

// ---------------------------------------------------------------------------
// Direct-to-LDS loads.  A buffer load with the LDS bit moves 16 bytes per
// lane from global memory straight into LDS: lane l of the instruction
// writes bytes [16 l, 16 l + 16) past its wave-uniform LDS base (held in
// M0), without passing through registers.  The compiler does not see that
// LDS write, so a wave waits for the load count (wait_vm) and the
// workgroup then synchronises before any wave reads those bytes.
// ---------------------------------------------------------------------------
typedef int i32x4 __attribute__((ext_vector_type(4)));
__device__ void raw_buffer_load_lds(i32x4 rsrc, __attribute__((address_space(3))) uint32_t* lds, int size,
                                    int voffset, int soffset, int offset,
                                    int aux) __asm("llvm.amdgcn.raw.buffer.load.lds");

// Buffer descriptor of a whole operand: base, size in bytes (below 2^31, so
// that the offset 2^31 used for rows outside the operand is past the end and
// reads zeros).
__device__ inline i32x4 buffer_rsrc(const void* base, uint32_t bytes) {
  const uint64_t b = (uint64_t)base;
  i32x4 r;
  r[0] = (int)(uint32_t)b;
  r[1] = (int)(uint32_t)(b >> 32);
  r[2] = (int)bytes;
  r[3] = 0x00020000;
  return r;
}

// Wait until at most N of this wave's vector-memory operations are
// outstanding (they complete in issue order).
template <int N>
__device__ inline void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Workgroup barrier for LDS hand-offs only: the wave's own LDS operations
// complete, then the barrier.  Unlike __syncthreads() it carries no memory
// fence, whose release half would make every wave wait for all of its
// outstanding global loads, the direct-to-LDS ones still meant to be in
// flight included.  Direct-to-LDS data a wave is about to hand over must be
// waited for with wait_vm first.
__device__ inline void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

}  // namespace terra
