// block.hip - the rest of one Swin block around the window attention
// (Sec. IV-A Swin blocks; Sec. IV-C: the linear layers that TP shards;
// Table III model widths): LayerNorm, the QKV projection, the output
// projection and the GELU MLP, forward and backward, bf16 storage with
// float32 accumulation.
//
// One matrix-core GEMM kernel serves every linear layer.  Operands are
// bf16 row-major matrices in HBM; each is staged through LDS in its memory
// layout, and its 32 x 16 matrix-core operands are read either straight
// (when the contraction index runs along memory rows) or through the LDS
// transpose read (when it runs down memory columns), so Y = X W^T,
// dX = dY W and dW = dY^T X all take the same kernel.  LayerNorm is applied
// to an operand while it is staged (from per-token mean and 1/std computed
// by a small kernel), so normalised activations never reach HBM; bias,
// residual, GELU and its derivative are applied in the epilogue.
#include "terra_common.h"
#include "terra_block.h"

namespace terra {

typedef __bf16 bf16;
typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;

constexpr int kGT = 256;          // threads per GEMM workgroup (4 waves, 2 x 2)
constexpr int kBM = 256;          // workgroup tile rows
constexpr int kBN = 128;          // workgroup tile columns
constexpr int kBK = 32;           // contraction depth per stage
constexpr int kPadR = 8;          // LDS row padding of contraction-contiguous tiles
constexpr int kPadC = 8;          // LDS row padding of contraction-strided tiles

// A bf16 operand in memory: row-major, split into up to three column blocks
// of `split` columns each (the Q, K and V tensors of the QKV layer are one
// operand of 3C columns held as three C-column tensors).  rows: valid rows.
struct Mat {
  const bf16* p[3];
  int split;
  int rows;
  __device__ const bf16* at(int r, int c) const {
    const int blk = c / split;
    return p[blk] + (int64_t)r * split + (c - blk * split);
  }
};

// LayerNorm of a staged operand: memory rows are tokens (mean, rstd),
// memory columns channels (gamma, beta).
struct LnArgs {
  const float* mean;
  const float* rstd;
  const float* gamma;
  const float* beta;
};

enum Epi {
  EPI_BIAS = 0,        // out = bf16(acc + bias)                (column-split output)
  EPI_BIAS_RES = 1,    // out = bf16(acc + bias + res)
  EPI_BIAS_GELU = 2,   // out = bf16(acc + bias), out2 = bf16(GELU(acc + bias))
  EPI_GELU_GRAD = 3,   // out = bf16(acc * GELU'(aux))
  EPI_F32 = 4,         // outf = acc (float32), slice blockIdx.z
  EPI_BF16 = 5,        // out = bf16(acc)
};

struct EpiArgs {
  bf16* out[3];        // column-split bf16 output (split columns each)
  int split;
  bf16* out2;          // second bf16 output (GELU), ld = N
  const bf16* aux;     // residual or pre-activation, ld = N
  const float* bias;
  float* outf;         // float32 output, ld = N, slice stride M * N
};

__device__ inline float gelu_f(float t) { return 0.5f * t * (1.0f + erff(t * 0.70710678118654752f)); }
__device__ inline float gelu_grad_f(float t) {
  return 0.5f * (1.0f + erff(t * 0.70710678118654752f)) + t * 0.39894228040143268f * __expf(-0.5f * t * t);
}

// Natural-order transposed operand from a tile stored [k][m] (row stride S):
// lane l receives T[k0 + 8h + x][m0 + l % 32], x = 0..7, h = l / 32.  In
// each 16-lane group G of the transpose read, lane i gets element i % 4 of
// the 8 bytes that lane 16G + 4x + i/4 addresses, so lane L addresses row
// k0 + 8h + (L % 16) / 4 (and 4 rows further for the second read), columns
// m0 + 16 (G % 2) + 4 (L % 4).
template <int S>
__device__ inline bf16x8 tr_operand(const bf16* T, int k0, int m0, int lane) {
  const int G = lane >> 4;
  const bf16* p = T + (k0 + 8 * (G >> 1) + ((lane & 15) >> 2)) * S + m0 + 16 * (G & 1) + 4 * (lane & 3);
  const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)p);
  const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(p + 4 * S));
  typedef short v8s __attribute__((ext_vector_type(8)));
  const v8s o = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, o);
}

// Straight operand from a tile stored [m][k] (row stride S): lane l
// receives T[m0 + l % 32][k0 + 8h + x].
template <int S>
__device__ inline bf16x8 row_operand(const bf16* T, int k0, int m0, int lane) {
  return *reinterpret_cast<const bf16x8*>(T + (m0 + (lane & 31)) * S + k0 + 8 * (lane >> 5));
}

// Staging geometry of one operand tile (R rows of the output side x kBK).
// KROW: the contraction index runs along memory rows (memory [R][kBK]);
// otherwise down memory columns (memory [kBK][R]).
template <int R, bool KROW>
struct Stage {
  static constexpr int kChunks = R * kBK / 8;                 // 16-byte chunks per stage
  static constexpr int kPer = kChunks / kGT;                  // per thread
  static constexpr int kS = KROW ? kBK + kPadR : R + kPadC;   // LDS row stride
  static constexpr int kElems = KROW ? R * kS : kBK * kS;
  // memory row / column of chunk c of the tile at (r0 output rows, k0)
  __device__ static void where(int c, int r0, int k0, int& mrow, int& mcol) {
    if (KROW) {
      mrow = r0 + c / (kBK / 8);
      mcol = k0 + 8 * (c % (kBK / 8));
    } else {
      mrow = k0 + c / (R / 8);
      mcol = r0 + 8 * (c % (R / 8));
    }
  }
  __device__ static int lds_off(int c) {
    if (KROW) return (c / (kBK / 8)) * kS + 8 * (c % (kBK / 8));
    return (c / (R / 8)) * kS + 8 * (c % (R / 8));
  }
};

template <bool LN>
__device__ inline uint4 ln_chunk(uint4 raw, const LnArgs& ln, int mrow, int mcol) {
  if (!LN) return raw;
  const float mu = ln.mean[mrow], rs = ln.rstd[mrow];
  const float4 g0 = *reinterpret_cast<const float4*>(ln.gamma + mcol);
  const float4 g1 = *reinterpret_cast<const float4*>(ln.gamma + mcol + 4);
  const float4 b0 = *reinterpret_cast<const float4*>(ln.beta + mcol);
  const float4 b1 = *reinterpret_cast<const float4*>(ln.beta + mcol + 4);
  const float g[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
  const float b[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
  bf16x8 v = __builtin_bit_cast(bf16x8, raw);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (bf16)(((float)v[i] - mu) * rs * g[i] + b[i]);
  return __builtin_bit_cast(uint4, v);
}

// C[M][N] = A[M][K] B[K][N] (+ epilogue).  AKROW: A is memory [M][K]
// (else [K][M]); BKROW: B is memory [N][K] (else [K][N]).  LNA / LNB:
// LayerNorm applied to A / B while staging (memory rows = tokens).
// blockIdx.z: contraction slice [z * kslice, (z+1) * kslice).
template <bool AKROW, bool BKROW, bool LNA, bool LNB, int EPI>
__global__ __launch_bounds__(kGT, 2) void gemm_kernel(Mat A, Mat B, LnArgs lna, LnArgs lnb, EpiArgs ep,
                                                      int M, int N, int K, int kslice) {
  typedef Stage<kBM, AKROW> SA;
  typedef Stage<kBN, BKROW> SB;
  extern __shared__ __align__(16) char smem[];
  bf16* la[2];
  bf16* lb[2];
  la[0] = reinterpret_cast<bf16*>(smem);
  la[1] = la[0] + SA::kElems;
  lb[0] = la[1] + SA::kElems;
  lb[1] = lb[0] + SB::kElems;

  const int nN = N / kBN;
  const int nM = (M + kBM - 1) / kBM;
  const int tiles = nM * nN;
  int w = blockIdx.x;
  if (tiles % 8 == 0) w = (blockIdx.x % 8) * (tiles / 8) + blockIdx.x / 8;   // same-XCD neighbours
  const int tm = w / nN, tn = w - (w / nN) * nN;
  const int m0 = tm * kBM, n0 = tn * kBN;
  const int kbeg = blockIdx.z * kslice;
  const int kend = min(K, kbeg + kslice);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = (wave >> 1) * 128, wn = (wave & 1) * 64;

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  uint4 ra[SA::kPer], rb[SB::kPer];
  auto load = [&](int k0) {
#pragma unroll
    for (int u = 0; u < SA::kPer; ++u) {
      int mr, mc;
      SA::where(threadIdx.x + u * kGT, m0, k0, mr, mc);
      const bool ok = AKROW ? (mr < M && mc < kend) : (mr < kend && mc < M);
      ra[u] = ok ? *reinterpret_cast<const uint4*>(A.at(mr, mc)) : make_uint4(0, 0, 0, 0);
      if (LNA && ok) ra[u] = ln_chunk<true>(ra[u], lna, mr, mc);
    }
#pragma unroll
    for (int u = 0; u < SB::kPer; ++u) {
      int mr, mc;
      SB::where(threadIdx.x + u * kGT, n0, k0, mr, mc);
      const bool ok = BKROW ? (mc < kend) : (mr < kend);
      rb[u] = ok ? *reinterpret_cast<const uint4*>(B.at(mr, mc)) : make_uint4(0, 0, 0, 0);
      if (LNB && ok) rb[u] = ln_chunk<true>(rb[u], lnb, mr, mc);
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int u = 0; u < SA::kPer; ++u)
      *reinterpret_cast<uint4*>(la[buf] + SA::lds_off(threadIdx.x + u * kGT)) = ra[u];
#pragma unroll
    for (int u = 0; u < SB::kPer; ++u)
      *reinterpret_cast<uint4*>(lb[buf] + SB::lds_off(threadIdx.x + u * kGT)) = rb[u];
  };

  const int nk = (kend - kbeg + kBK - 1) / kBK;
  if (nk > 0) {
    load(kbeg);
    store(0);
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load(kbeg + (kt + 1) * kBK);
#pragma unroll
    for (int c = 0; c < kBK / 16; ++c) {
      bf16x8 bo[2];
#pragma unroll
      for (int j = 0; j < 2; ++j)
        bo[j] = BKROW ? row_operand<SB::kS>(lb[buf], 16 * c, wn + 32 * j, lane)
                      : tr_operand<SB::kS>(lb[buf], 16 * c, wn + 32 * j, lane);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bf16x8 ao = AKROW ? row_operand<SA::kS>(la[buf], 16 * c, wm + 32 * i, lane)
                                : tr_operand<SA::kS>(la[buf], 16 * c, wm + 32 * i, lane);
#pragma unroll
        for (int j = 0; j < 2; ++j) mma16(acc[i][j], ao, bo[j]);
      }
    }
    if (kt + 1 < nk) store(buf ^ 1);
    __syncthreads();
  }

  // Epilogue.  acc[i][j] holds rows wm + 32i + 8g + 4h + x (register 4g + x),
  // column wn + 32j + lane % 32.
  const int h = lane >> 5, col = lane & 31;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int n = n0 + wn + 32 * j + col;
    const float bias = (EPI == EPI_BIAS || EPI == EPI_BIAS_RES || EPI == EPI_BIAS_GELU) ? ep.bias[n] : 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm + 32 * i + 8 * (r / 4) + 4 * h + (r % 4);
        if (m >= M) continue;
        const float v = acc[i][j][r];
        const int64_t o = (int64_t)m * N + n;
        if (EPI == EPI_BIAS) {
          const int blk = n / ep.split;
          ep.out[blk][(int64_t)m * ep.split + (n - blk * ep.split)] = (bf16)(v + bias);
        } else if (EPI == EPI_BIAS_RES) {
          ep.out[0][o] = (bf16)(v + bias + (float)ep.aux[o]);
        } else if (EPI == EPI_BIAS_GELU) {
          const float t = v + bias;
          ep.out[0][o] = (bf16)t;
          ep.out2[o] = (bf16)gelu_f(t);
        } else if (EPI == EPI_GELU_GRAD) {
          ep.out[0][o] = (bf16)(v * gelu_grad_f((float)ep.aux[o]));
        } else if (EPI == EPI_F32) {
          ep.outf[(int64_t)blockIdx.z * M * N + o] = v;
        } else {
          ep.out[0][o] = (bf16)v;
        }
      }
  }
}

// ---------------------------------------------------------------------------
// LayerNorm statistics: one wave per token, mean and 1 / sqrt(var + eps)
// (biased variance, two passes over the row).
// ---------------------------------------------------------------------------
constexpr int kRowThreads = 256;

__device__ inline float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

__global__ __launch_bounds__(kRowThreads) void ln_stats_kernel(const bf16* __restrict__ x, float* __restrict__ mean,
                                                               float* __restrict__ rstd, int T, int C, float eps) {
  const int row = blockIdx.x * (kRowThreads / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= T) return;
  const bf16* p = x + (int64_t)row * C;
  float s = 0.0f;
  for (int c = 8 * lane; c < C; c += 512) {
    const bf16x8 v = *reinterpret_cast<const bf16x8*>(p + c);
#pragma unroll
    for (int i = 0; i < 8; ++i) s += (float)v[i];
  }
  const float mu = wave_sum(s) / (float)C;
  float q = 0.0f;
  for (int c = 8 * lane; c < C; c += 512) {
    const bf16x8 v = *reinterpret_cast<const bf16x8*>(p + c);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float d = (float)v[i] - mu;
      q += d * d;
    }
  }
  const float var = wave_sum(q) / (float)C;
  if (lane == 0) {
    mean[row] = mu;
    rstd[row] = 1.0f / sqrtf(var + eps);
  }
}

// ---------------------------------------------------------------------------
// LayerNorm backward plus the residual branch, one wave per token:
//   g = dy * gamma, dz = rstd (g - mean(g) - zhat mean(g zhat)) + dres
// written as bf16; per-wave partial sums of dy * zhat (dgamma) and dy
// (dbeta) over the wave's tokens go to `part` ([wave][2][C]) for a
// fixed-order reduction.  Each lane owns channel chunks 8 (lane + 64 c).
// ---------------------------------------------------------------------------
constexpr int kLnMaxChunks = 4;   // C <= 4 * 512 = 2048

__global__ __launch_bounds__(kRowThreads) void ln_bwd_kernel(
    const float* __restrict__ dy, const bf16* __restrict__ z, const float* __restrict__ mean,
    const float* __restrict__ rstd, const float* __restrict__ gamma, const bf16* __restrict__ dres,
    bf16* __restrict__ dz, float* __restrict__ part, int T, int C, int rows_per_wave) {
  const int gw = blockIdx.x * (kRowThreads / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  float dg[kLnMaxChunks][8], db[kLnMaxChunks][8];
#pragma unroll
  for (int c = 0; c < kLnMaxChunks; ++c)
#pragma unroll
    for (int i = 0; i < 8; ++i) dg[c][i] = db[c][i] = 0.0f;
  const int r0 = gw * rows_per_wave;
  const int r1 = min(T, r0 + rows_per_wave);
  const float invC = 1.0f / (float)C;
  for (int row = r0; row < r1; ++row) {
    const float mu = mean[row], rs = rstd[row];
    float zh[kLnMaxChunks][8], gg[kLnMaxChunks][8];
    float s1 = 0.0f, s2 = 0.0f;
#pragma unroll
    for (int c = 0; c < kLnMaxChunks; ++c) {
      const int ch = 8 * (lane + 64 * c);
      if (ch < C) {
        const bf16x8 zv = *reinterpret_cast<const bf16x8*>(z + (int64_t)row * C + ch);
        const float4 d0 = *reinterpret_cast<const float4*>(dy + (int64_t)row * C + ch);
        const float4 d1 = *reinterpret_cast<const float4*>(dy + (int64_t)row * C + ch + 4);
        const float d[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          zh[c][i] = ((float)zv[i] - mu) * rs;
          gg[c][i] = d[i] * gamma[ch + i];
          s1 += gg[c][i];
          s2 += gg[c][i] * zh[c][i];
          dg[c][i] += d[i] * zh[c][i];
          db[c][i] += d[i];
        }
      }
    }
    s1 = wave_sum(s1) * invC;
    s2 = wave_sum(s2) * invC;
#pragma unroll
    for (int c = 0; c < kLnMaxChunks; ++c) {
      const int ch = 8 * (lane + 64 * c);
      if (ch < C) {
        const bf16x8 rv = *reinterpret_cast<const bf16x8*>(dres + (int64_t)row * C + ch);
        bf16x8 o;
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] = (bf16)(rs * (gg[c][i] - s1 - zh[c][i] * s2) + (float)rv[i]);
        *reinterpret_cast<bf16x8*>(dz + (int64_t)row * C + ch) = o;
      }
    }
  }
  float* pg = part + (int64_t)gw * 2 * C;
#pragma unroll
  for (int c = 0; c < kLnMaxChunks; ++c) {
    const int ch = 8 * (lane + 64 * c);
    if (ch < C) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        pg[ch + i] = dg[c][i];
        pg[C + ch + i] = db[c][i];
      }
    }
  }
}

// Column sums of a (column-split) bf16 matrix, per slice of rows:
// part[s][col] = sum over rows [s * rows_per, (s+1) * rows_per) - the bias
// gradients, reduced afterwards in slice order.  Thread = 8 columns.
__global__ __launch_bounds__(kRowThreads) void colsum_kernel(Mat X, int ncols, float* __restrict__ part,
                                                             int rows_per) {
  const int c8 = blockIdx.x * kRowThreads + threadIdx.x;
  if (8 * c8 >= ncols) return;
  const int s = blockIdx.y;
  const int r0 = s * rows_per, r1 = min(X.rows, r0 + rows_per);
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int r = r0; r < r1; ++r) {
    const bf16x8 v = *reinterpret_cast<const bf16x8*>(X.at(r, 8 * c8));
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] += (float)v[i];
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) part[(int64_t)s * ncols + 8 * c8 + i] = acc[i];
}

// out[i] = sum over s < nslice of part[s * stride + i], in slice order.
__global__ __launch_bounds__(kRowThreads) void slice_sum_kernel(const float* __restrict__ part, float* __restrict__ out,
                                                                int64_t n, int64_t stride, int nslice) {
  const int64_t i = (int64_t)blockIdx.x * kRowThreads + threadIdx.x;
  if (i >= n) return;
  float acc = 0.0f;
  for (int s = 0; s < nslice; ++s) acc += part[(int64_t)s * stride + i];
  out[i] = acc;
}

// ---------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------
static size_t gemm_lds(bool akrow, bool bkrow) {
  const size_t a = akrow ? (size_t)kBM * (kBK + kPadR) : (size_t)kBK * (kBM + kPadC);
  const size_t b = bkrow ? (size_t)kBN * (kBK + kPadR) : (size_t)kBK * (kBN + kPadC);
  return 2 * (a + b) * sizeof(bf16);
}

template <bool AKROW, bool BKROW, bool LNA, bool LNB, int EPI>
static hipError_t gemm(const Mat& A, const Mat& B, const LnArgs& lna, const LnArgs& lnb, const EpiArgs& ep,
                       int M, int N, int K, int nsplit, hipStream_t st) {
  const int tiles = ((M + kBM - 1) / kBM) * (N / kBN);
  const int kslice = ((K + nsplit - 1) / nsplit + kBK - 1) / kBK * kBK;
  hipLaunchKernelGGL((gemm_kernel<AKROW, BKROW, LNA, LNB, EPI>), dim3(tiles, 1, nsplit), dim3(kGT),
                     gemm_lds(AKROW, BKROW), st, A, B, lna, lnb, ep, M, N, K, kslice);
  return hipGetLastError();
}

static Mat mat(const void* p, int split, int rows) {
  Mat m;
  m.p[0] = m.p[1] = m.p[2] = (const bf16*)p;
  m.split = split;
  m.rows = rows;
  return m;
}
static Mat mat3(const void* p0, const void* p1, const void* p2, int split, int rows) {
  Mat m;
  m.p[0] = (const bf16*)p0;
  m.p[1] = (const bf16*)p1;
  m.p[2] = (const bf16*)p2;
  m.split = split;
  m.rows = rows;
  return m;
}

constexpr float kLnEps = 1e-5f;

hipError_t launch_attn_fwd(const Geo& g, int dt, bool nhwc, const void* q, const void* k, const void* v,
                           const float* table, void* o, float* lse, hipStream_t st);
hipError_t launch_attn_bwd(const Geo& g, int dt, bool nhwc, const void* q, const void* k, const void* v,
                           const void* o, const void* dout, const float* lse, const float* table, void* dq,
                           void* dk, void* dv, float* dtab, void* ws, hipStream_t st);
size_t bwd_workspace(const Geo& g, int dt);

static hipError_t ln_stats(const void* x, float* mu, float* rs, int T, int C, hipStream_t st) {
  const int per = kRowThreads / 64;
  hipLaunchKernelGGL(ln_stats_kernel, dim3((T + per - 1) / per), dim3(kRowThreads), 0, st, (const bf16*)x, mu, rs,
                     T, C, kLnEps);
  return hipGetLastError();
}

hipError_t launch_block_fwd(const Geo& g, const void* x, const BlockParams& p, const float* table, void* x2,
                            const BlockSaved& s, hipStream_t st) {
  const int T = g.B * g.H * g.W, C = g.C;
  hipError_t e;
  LnArgs none = {nullptr, nullptr, nullptr, nullptr};
  EpiArgs ep = {};
  // LN1 statistics, then qkv = LN1(x) W_qkv^T + b_qkv into Q, K, V (NHWC)
  if ((e = ln_stats(x, s.mu1, s.rstd1, T, C, st)) != hipSuccess) return e;
  LnArgs ln1 = {s.mu1, s.rstd1, p.ln1_g, p.ln1_b};
  ep.out[0] = (bf16*)s.q; ep.out[1] = (bf16*)s.k; ep.out[2] = (bf16*)s.v; ep.split = C;
  ep.bias = p.b_qkv;
  if ((e = gemm<true, true, true, false, EPI_BIAS>(mat(x, C, T), mat(p.w_qkv, C, 3 * C), ln1, none, ep, T, 3 * C,
                                                   C, 1, st)) != hipSuccess)
    return e;
  // windowed attention with the route fused in
  if ((e = launch_attn_fwd(g, 1, true, s.q, s.k, s.v, table, s.o, s.lse, st)) != hipSuccess) return e;
  // x1 = x + o W_p^T + b_p
  ep = EpiArgs{};
  ep.out[0] = (bf16*)s.x1; ep.split = C; ep.aux = (const bf16*)x; ep.bias = p.b_proj;
  if ((e = gemm<true, true, false, false, EPI_BIAS_RES>(mat(s.o, C, T), mat(p.w_proj, C, C), none, none, ep, T, C,
                                                        C, 1, st)) != hipSuccess)
    return e;
  // h = LN2(x1) W_1^T + b_1, a = GELU(h)
  if ((e = ln_stats(s.x1, s.mu2, s.rstd2, T, C, st)) != hipSuccess) return e;
  LnArgs ln2 = {s.mu2, s.rstd2, p.ln2_g, p.ln2_b};
  ep = EpiArgs{};
  ep.out[0] = (bf16*)s.h; ep.split = 4 * C; ep.out2 = (bf16*)s.a; ep.bias = p.b_fc1;
  if ((e = gemm<true, true, true, false, EPI_BIAS_GELU>(mat(s.x1, C, T), mat(p.w_fc1, C, 4 * C), ln2, none, ep, T,
                                                         4 * C, C, 1, st)) != hipSuccess)
    return e;
  // x2 = x1 + a W_2^T + b_2
  ep = EpiArgs{};
  ep.out[0] = (bf16*)x2; ep.split = C; ep.aux = (const bf16*)s.x1; ep.bias = p.b_fc2;
  return gemm<true, true, false, false, EPI_BIAS_RES>(mat(s.a, 4 * C, T), mat(p.w_fc2, 4 * C, C), none, none, ep, T,
                                                      C, 4 * C, 1, st);
}

// Backward workspace layout (bytes, 256-aligned pieces).
struct BwdWs {
  size_t dh, dln, dx1, dO, dq, dk, dv, attn, wpart, cpart, lpart, total;
  int wsplit, cslices, lnwaves, rows_per_wave, cpart_rows;
};

static size_t al(size_t x) { return (x + 255) / 256 * 256; }

// A pure function of the geometry: the attention part is sized for kMaxCus
// whatever device the call runs on.
static BwdWs block_ws(const Geo& geo) {
  Geo g = geo;
  g.cus = kMaxCus;
  BwdWs w;
  const size_t T = (size_t)g.B * g.H * g.W, C = g.C;
  w.wsplit = 16;                         // contraction (token) slices of the weight gradients
  w.cslices = 512;                       // row slices of the bias-gradient column sums
  w.cpart_rows = (int)((T + w.cslices - 1) / w.cslices);
  w.lnwaves = 2048;                      // waves of the LayerNorm backward
  w.rows_per_wave = (int)((T + w.lnwaves - 1) / w.lnwaves);
  size_t off = 0;
  w.dh = off; off += al(T * 4 * C * 2);
  w.dln = off; off += al(T * C * 4);
  w.dx1 = off; off += al(T * C * 2);
  w.dO = off; off += al(T * C * 2);
  w.dq = off; off += al(T * C * 2);
  w.dk = off; off += al(T * C * 2);
  w.dv = off; off += al(T * C * 2);
  w.attn = off; off += al(bwd_workspace(g, 1));
  w.wpart = off; off += al((size_t)w.wsplit * 4 * C * C * 4);
  w.cpart = off; off += al((size_t)w.cslices * 4 * C * 4);
  w.lpart = off; off += al((size_t)w.lnwaves * 2 * C * 4);
  w.total = off;
  return w;
}

size_t block_bwd_workspace(const Geo& g) { return block_ws(g).total; }

static hipError_t slice_sum(const float* part, float* out, int64_t n, int nslice, hipStream_t st,
                            int64_t stride = -1) {
  hipLaunchKernelGGL(slice_sum_kernel, dim3((unsigned)((n + kRowThreads - 1) / kRowThreads)), dim3(kRowThreads), 0,
                     st, part, out, n, stride < 0 ? n : stride, nslice);
  return hipGetLastError();
}

// LayerNorm parameter gradients from the per-wave partials [wave][dgamma C | dbeta C].
static hipError_t ln_param_grads(const float* lpart, float* dgamma, float* dbeta, int C, int nwaves, hipStream_t st) {
  hipError_t e = slice_sum(lpart, dgamma, C, nwaves, st, 2 * C);
  if (e != hipSuccess) return e;
  return slice_sum(lpart + C, dbeta, C, nwaves, st, 2 * C);
}

static hipError_t colsum(const Mat& X, int ncols, float* part, float* out, const BwdWs& w, hipStream_t st) {
  hipLaunchKernelGGL(colsum_kernel, dim3((ncols / 8 + kRowThreads - 1) / kRowThreads, w.cslices), dim3(kRowThreads),
                     0, st, X, ncols, part, w.cpart_rows);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return slice_sum(part, out, ncols, w.cslices, st);
}

// Weight gradient dW[Nl][Kl] = dY^T Z over all tokens (dY: T x Nl, Z: T x Kl),
// in token slices, reduced in slice order.  LNB: Z = LN(z) applied on the fly.
template <bool LNB>
static hipError_t wgrad(const Mat& dY, const Mat& Z, const LnArgs& ln, int T, int Nl, int Kl, float* dW,
                        char* ws, const BwdWs& w, hipStream_t st) {
  LnArgs none = {nullptr, nullptr, nullptr, nullptr};
  EpiArgs ep = {};
  float* part = reinterpret_cast<float*>(ws + w.wpart);
  ep.outf = part;
  hipError_t e = gemm<false, false, false, LNB, EPI_F32>(dY, Z, none, ln, ep, Nl, Kl, T, w.wsplit, st);
  if (e != hipSuccess) return e;
  return slice_sum(part, dW, (int64_t)Nl * Kl, w.wsplit, st);
}

hipError_t launch_block_bwd(const Geo& g, const void* dx2, const void* x, const BlockParams& p, const float* table,
                            const BlockSaved& s, void* dx, const BlockGrads& gr, float* dtable, void* wsv,
                            hipStream_t st) {
  const int T = g.B * g.H * g.W, C = g.C;
  const BwdWs w = block_ws(g);
  char* ws = reinterpret_cast<char*>(wsv);
  bf16* dh = reinterpret_cast<bf16*>(ws + w.dh);
  float* dln = reinterpret_cast<float*>(ws + w.dln);
  bf16* dx1 = reinterpret_cast<bf16*>(ws + w.dx1);
  bf16* dO = reinterpret_cast<bf16*>(ws + w.dO);
  bf16* dq = reinterpret_cast<bf16*>(ws + w.dq);
  bf16* dk = reinterpret_cast<bf16*>(ws + w.dk);
  bf16* dv = reinterpret_cast<bf16*>(ws + w.dv);
  float* cpart = reinterpret_cast<float*>(ws + w.cpart);
  float* lpart = reinterpret_cast<float*>(ws + w.lpart);
  LnArgs none = {nullptr, nullptr, nullptr, nullptr};
  hipError_t e;
  EpiArgs ep = {};
#define TERRA_TRY(x) \
  if ((e = (x)) != hipSuccess) return e
  // x2 = x1 + a W2^T + b2:  dW2 = dx2^T a, db2 = colsum(dx2), dh = (dx2 W2) * GELU'(h)
  TERRA_TRY(wgrad<false>(mat(dx2, C, T), mat(s.a, 4 * C, T), none, T, C, 4 * C, gr.w_fc2, ws, w, st));
  TERRA_TRY(colsum(mat(dx2, C, T), C, cpart, gr.b_fc2, w, st));
  ep.out[0] = dh; ep.split = 4 * C; ep.aux = (const bf16*)s.h;
  TERRA_TRY((gemm<true, false, false, false, EPI_GELU_GRAD>(mat(dx2, C, T), mat(p.w_fc2, 4 * C, C), none, none, ep,
                                                             T, 4 * C, C, 1, st)));
  // h = LN2(x1) W1^T + b1:  dW1 = dh^T LN2(x1), db1 = colsum(dh), dln2 = dh W1
  LnArgs ln2 = {s.mu2, s.rstd2, p.ln2_g, p.ln2_b};
  TERRA_TRY(wgrad<true>(mat(dh, 4 * C, T), mat(s.x1, C, T), ln2, T, 4 * C, C, gr.w_fc1, ws, w, st));
  TERRA_TRY(colsum(mat(dh, 4 * C, T), 4 * C, cpart, gr.b_fc1, w, st));
  ep = EpiArgs{};
  ep.outf = dln;
  TERRA_TRY((gemm<true, false, false, false, EPI_F32>(mat(dh, 4 * C, T), mat(p.w_fc1, C, 4 * C), none, none, ep, T,
                                                       C, 4 * C, 1, st)));
  // dx1 = dx2 + LN2 backward
  hipLaunchKernelGGL(ln_bwd_kernel, dim3(w.lnwaves / 4), dim3(kRowThreads), 0, st, dln, (const bf16*)s.x1, s.mu2,
                     s.rstd2, p.ln2_g, (const bf16*)dx2, dx1, lpart, T, C, w.rows_per_wave);
  TERRA_TRY(hipGetLastError());
  TERRA_TRY(ln_param_grads(lpart, gr.ln2_g, gr.ln2_b, C, w.lnwaves, st));
  // x1 = x + o Wp^T + bp:  dWp = dx1^T o, dbp = colsum(dx1), dO = dx1 Wp
  TERRA_TRY(wgrad<false>(mat(dx1, C, T), mat(s.o, C, T), none, T, C, C, gr.w_proj, ws, w, st));
  TERRA_TRY(colsum(mat(dx1, C, T), C, cpart, gr.b_proj, w, st));
  ep = EpiArgs{};
  ep.out[0] = dO; ep.split = C;
  TERRA_TRY((gemm<true, false, false, false, EPI_BF16>(mat(dx1, C, T), mat(p.w_proj, C, C), none, none, ep, T, C, C,
                                                        1, st)));
  // attention backward (route fused in)
  TERRA_TRY(launch_attn_bwd(g, 1, true, s.q, s.k, s.v, s.o, dO, s.lse, table, dq, dk, dv, dtable, ws + w.attn, st));
  // qkv = LN1(x) Wqkv^T + bqkv:  dWqkv = dqkv^T LN1(x), dbqkv, dln1 = dqkv Wqkv
  LnArgs ln1 = {s.mu1, s.rstd1, p.ln1_g, p.ln1_b};
  const Mat dqkv = mat3(dq, dk, dv, C, T);
  TERRA_TRY(wgrad<true>(dqkv, mat(x, C, T), ln1, T, 3 * C, C, gr.w_qkv, ws, w, st));
  TERRA_TRY(colsum(dqkv, 3 * C, cpart, gr.b_qkv, w, st));
  ep = EpiArgs{};
  ep.outf = dln;
  TERRA_TRY((gemm<true, false, false, false, EPI_F32>(dqkv, mat(p.w_qkv, C, 3 * C), none, none, ep, T, C, 3 * C, 1,
                                                       st)));
  // dx = dx1 + LN1 backward
  hipLaunchKernelGGL(ln_bwd_kernel, dim3(w.lnwaves / 4), dim3(kRowThreads), 0, st, dln, (const bf16*)x, s.mu1,
                     s.rstd1, p.ln1_g, (const bf16*)dx1, (bf16*)dx, lpart, T, C, w.rows_per_wave);
  TERRA_TRY(hipGetLastError());
  TERRA_TRY(ln_param_grads(lpart, gr.ln1_g, gr.ln1_b, C, w.lnwaves, st));
#undef TERRA_TRY
  return hipSuccess;
}

}  // namespace terra
