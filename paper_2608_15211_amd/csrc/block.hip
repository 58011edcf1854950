// block.hip - the rest of one Swin block around the window attention
// (Sec. IV-A Swin blocks; Sec. IV-C: the linear layers that TP shards;
// Table III model widths): LayerNorm, the QKV projection, the output
// projection and the GELU MLP, forward and backward, bf16 storage with
// float32 accumulation.
//
// One matrix-core GEMM kernel serves every linear layer.  Operands are
// bf16 row-major matrices in HBM, brought into XOR-swizzled LDS tiles by
// direct-to-LDS loads through a three-stage ring; the 32 x 16 matrix-core
// operands are read either straight (when the contraction index runs along
// memory rows) or through the LDS transpose read (when it runs down memory
// columns), so Y = X W^T, dX = dY W and dW = dY^T X all take the same
// kernel.  In the forward each LayerNorm is folded into the projection
// after it (gains into the weights, mean and 1/std applied to the
// accumulators), so normalised activations never reach HBM there; the
// backward recomputes them once per weight gradient.  Bias, residual,
// GELU and its derivative are applied in the epilogue.
#include <algorithm>

#include "terra_common.h"
#include "terra_block.h"

namespace terra {

typedef __bf16 bf16;
typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;

constexpr int kGT = 512;          // threads per GEMM workgroup (8 waves: 2 rows x 4 columns of 128 x 64)
constexpr int kBM = 256;          // workgroup tile rows
constexpr int kBN = 256;          // workgroup tile columns (128 in the four-wave form)
constexpr int kBK = 32;           // contraction depth per stage
constexpr int kEpiS = 68;         // row stride (floats) of a wave's epilogue staging tile
constexpr int kMaxCusBlock = 256;  // compute units the weight-gradient slices are sized for

// A bf16 operand in memory: row-major, `ld` elements a row, `rows` valid rows.
struct Mat {
  const bf16* p;
  int ld;
  int rows;
  // Three-part operand (read only by SEG kernels): three [rows][segw]
  // matrices side by side, part i at element offset i * segstride from p.
  int segw;
  int64_t segstride;
  __device__ const bf16* at(int r, int c) const { return p + (int64_t)r * ld + c; }
};


enum Epi {
  EPI_LN_QKV = 0,      // LayerNorm folded: out = bf16(rstd (acc - mean s) + c)   (column-split output)
  EPI_BIAS_RES = 1,    // out = bf16(acc + bias + res)
  EPI_LN_GELU = 2,     // t = rstd (acc - mean s) + c:  out = bf16(t), out2 = bf16(GELU(t))
  EPI_GELU_GRAD = 3,   // out = bf16(acc * GELU'(aux))
  EPI_F32 = 4,         // outf = acc (float32), slice blockIdx.z
  EPI_BF16 = 5,        // out = bf16(acc)
  EPI_F32_ACC = 6,     // outf += acc (float32)
};

struct EpiArgs {
  bf16* out[3];        // column-split bf16 output (split columns each)
  int split;
  bf16* out2;          // second bf16 output (GELU), ld = N
  const bf16* aux;     // residual or pre-activation, ld = N
  const float* bias;
  float* outf;         // float32 output, ld = N, slice stride M * N
  const float* mean;   // LayerNorm folded into the epilogue: per-row mean and 1/std,
  const float* rstd;   // per-column sum of the folded weights (lns) and constant (lnc)
  const float* lns;
  const float* lnc;
  // EPI_GELU_GRAD: column sums of the bf16 output over each wave's 128 rows,
  // partial row 2 (tile row) + (wave row), ld = N (nullable)
  float* colpart;
};

// Phi(x), the standard normal distribution function, and exp(-x^2 / 2), with
// erf from Abramowitz and Stegun's rational approximation 7.1.26
// (|error| <= 1.5e-7, far below bf16 resolution); the Gaussian factor is
// shared between erf and the GELU derivative.
__device__ inline void phi_gauss(float x, float& Phi, float& gauss) {
  const float z = fabsf(x) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(1.0f + 0.3275911f * z);
  gauss = __expf(-0.5f * x * x);
  const float poly =
      t * (0.254829592f + t * (-0.284496736f + t * (1.421413741f + t * (-1.453152027f + t * 1.061405429f))));
  const float erfz = 1.0f - poly * gauss;
  Phi = 0.5f * (1.0f + copysignf(erfz, x));
}
__device__ inline float gelu_f(float x) {
  float Phi, g;
  phi_gauss(x, Phi, g);
  return x * Phi;
}
__device__ inline float gelu_grad_f(float x) {
  float Phi, g;
  phi_gauss(x, Phi, g);
  return Phi + x * 0.39894228040143268f * g;   // Phi(x) + x phi(x)
}

// ---------------------------------------------------------------------------
// LDS tiles.  A stage holds the A tile (kBM output rows x kBK) and the B tile
// (kBN x kBK), each in its memory layout, unpadded, with the 16-byte chunks
// of each row permuted by an XOR of the row index so that the matrix-core
// operand reads hit distinct banks:
// * KROW tile (memory [R][kBK], 4 chunks a row): chunk c of row r sits at
//   chunk c ^ ((r >> 2) & 3) - 16 consecutive rows read at one logical chunk
//   cover all 64 banks;
// * COLK tile (memory [kBK][R], R / 8 chunks a row): chunk c of row k sits
//   at chunk c ^ (4 (k & 3)) - each half-wave of a transpose read takes 64
//   bytes from each of four rows, and these land on four different 64-byte
//   spans of the 256 bytes the LDS banks cover (measured: no bank conflicts;
//   with c ^ (2 (k & 3)) 0.8-2 conflict cycles per LDS instruction, though
//   no slower).
// ---------------------------------------------------------------------------
template <int R, bool KROW, int NT = kGT>
struct Tile {
  static constexpr int kChunks = R * kBK / 8;   // 16-byte chunks
  static constexpr int kPer = kChunks / NT;     // per thread (NT threads)
  static constexpr int kElems = R * kBK;
  // element offset of (row, logical chunk) of the memory layout
  __device__ static int off(int row, int c) {
    if (KROW) return row * kBK + 8 * (c ^ ((row >> 2) & 3));
    return row * R + 8 * (c ^ (4 * (row & 3)));
  }
  // memory (row, column) of the chunk stored in slot q (slot = chunk position in LDS order)
  __device__ static void slot_src(int q, int r0, int k0, int& mrow, int& mcol) {
    if (KROW) {
      const int row = q >> 2, p = q & 3;
      mrow = r0 + row;
      mcol = k0 + 8 * (p ^ ((row >> 2) & 3));
    } else {
      const int row = q / (R / 8), p = q - row * (R / 8);
      mrow = k0 + row;
      mcol = r0 + 8 * (p ^ (4 * (row & 3)));
    }
  }
};

// Straight operand (KROW tile): lane l receives T[m0 + l % 32][k0 + 8h + x],
// x = 0..7, h = l / 32, as one 16-byte read.
template <int R>
__device__ inline bf16x8 row_operand(const bf16* T, int k0, int m0, int lane) {
  const int row = m0 + (lane & 31);
  return *reinterpret_cast<const bf16x8*>(T + Tile<R, true>::off(row, (k0 >> 3) + (lane >> 5)));
}

// Natural-order transposed operand (COLK tile): lane l receives
// T[k0 + 8h + x][m0 + l % 32], x = 0..7.  In each 16-lane group G of the
// transpose read, lane i gets element i % 4 of the 8 bytes that lane
// 16G + 4x + i/4 addresses, so lane L addresses row k0 + 8h + (L % 16) / 4
// (4 rows further for the second read), columns m0 + 16 (G % 2) + 4 (L % 4).
template <int R>
__device__ inline bf16x8 tr_operand(const bf16* T, int k0, int m0, int lane) {
  const int G = lane >> 4;
  const int row = k0 + 8 * (G >> 1) + ((lane & 15) >> 2);
  const int m = m0 + 16 * (G & 1) + 4 * (lane & 3);
  const int c = m >> 3, e = m & 7;
  const bf16* p0 = T + Tile<R, false>::off(row, c) + e;
  const bf16* p1 = T + Tile<R, false>::off(row + 4, c) + e;
  const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)p0);
  const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)p1);
  typedef short v8s __attribute__((ext_vector_type(8)));
  const v8s o = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, o);
}

// Direct-to-LDS staging of one operand tile: each thread moves kPer 16-byte
// chunks with buffer loads that write LDS themselves (slot q of the tile is
// written by thread q % kGT, load q / kGT); chunks outside the operand or
// the contraction slice read zeros.  KROW: the contraction index runs along
// memory rows.
template <int R, bool KROW, int NT = kGT>
__device__ inline void stage_direct(const i32x4& rs, const Mat& X, bf16* tile, int r0, int k0, int nouter,
                                    int kend, int64_t base = 0) {
  typedef Tile<R, KROW, NT> T;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // uniform: the LDS base goes to M0
#pragma unroll
  for (int u = 0; u < T::kPer; ++u) {
    const int q = u * NT + threadIdx.x;
    int mr, mc;
    T::slot_src(q, r0, k0, mr, mc);
    const bool ok = KROW ? (mr < nouter && mc < kend) : (mr < kend && mc < nouter);
    const int voff = ok ? (int)((base + (int64_t)mr * X.ld + mc) * 2) : (int)0x80000000;
    bf16* dst = tile + 8 * (u * NT + wave * 64);       // wave-uniform base of 64 slots
    raw_buffer_load_lds(rs, (__attribute__((address_space(3))) uint32_t*)(uintptr_t)(uint32_t)(uintptr_t)dst, 16,
                        voff, 0, 0, 0);
  }
}


// C[M][N] = A[M][K] B[K][N] (+ epilogue).  AKROW: A is memory [M][K]
// (else [K][M]); BKROW: B is memory [N][K] (else [K][N]).  blockIdx.z:
// contraction slice [z * kslice, (z+1) * kslice).  Three LDS stages: the
// loads of stage kt + 2 are in flight while stage kt is on the matrix
// cores.  Eight waves, each a 128 x 64 block of the 256 x 256 tile.
// SEG: A is a three-part operand split along K (AKROW; A.segw a multiple of
// kBK) or along M (else; A.segw a multiple of kBM), so that every stage
// (AKROW) or every workgroup tile (else) reads one part.
// NW = 4: four waves and a 256 x 128 tile (72 KB of stages), so that two
// workgroups share a CU and one's prologue and epilogue (its operand
// latency, output traffic and, for some epilogues, input traffic) overlap
// the other's matrix work; for short contractions, where that per-tile time
// is a large part of the whole.
template <bool AKROW, bool BKROW, int EPI, bool SEG = false, int NW = 8>
__global__ __launch_bounds__(NW * 64, 8 / NW) void gemm_kernel(Mat A, Mat B, EpiArgs ep, int M, int N, int K,
                                                                int kslice) {
  constexpr int NT = NW * 64, BN = NW * 32;
  typedef Tile<kBM, AKROW, NT> TA;
  typedef Tile<BN, BKROW, NT> TB;
  constexpr int kStage = TA::kElems + TB::kElems;
  constexpr int kLoads = TA::kPer + TB::kPer;
  extern __shared__ __align__(16) char smem[];
  bf16* lds = reinterpret_cast<bf16*>(smem);

  const int nN = (N + BN - 1) / BN;
  const int nM = (M + kBM - 1) / kBM;
  const int tiles = nM * nN;
  int w = blockIdx.x;
  if (tiles % 8 == 0) w = (blockIdx.x % 8) * (tiles / 8) + blockIdx.x / 8;   // same-XCD neighbours
  const int tm = w / nN, tn = w - (w / nN) * nN;
  const int m0 = tm * kBM, n0 = tn * BN;
  const int kbeg = blockIdx.z * kslice;
  const int kend = min(K, kbeg + kslice);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = (wave / (NW / 2)) * 128, wn = (wave % (NW / 2)) * 64;
  const i32x4 rsa = buffer_rsrc(A.p, (uint32_t)(((int64_t)A.rows * A.ld + (SEG ? 2 * A.segstride : 0)) * 2));
  const i32x4 rsb = buffer_rsrc(B.p, (uint32_t)((int64_t)B.rows * B.ld * 2));

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  auto a_tile = [&](int st) { return lds + st * kStage; };
  auto b_tile = [&](int st) { return lds + st * kStage + TA::kElems; };
  auto issue = [&](int s) {
    const int k0 = kbeg + s * kBK;
    if constexpr (SEG && AKROW) {
      const int seg = k0 / A.segw;
      stage_direct<kBM, true, NT>(rsa, A, a_tile(s % 3), m0, k0 - seg * A.segw, M,
                                  min(kend - seg * A.segw, A.segw), seg * A.segstride);
    } else if constexpr (SEG) {
      const int seg = m0 / A.segw;
      stage_direct<kBM, false, NT>(rsa, A, a_tile(s % 3), m0 - seg * A.segw, k0, min(M - seg * A.segw, A.segw),
                                   kend, seg * A.segstride);
    } else {
      stage_direct<kBM, AKROW, NT>(rsa, A, a_tile(s % 3), m0, k0, M, kend);
    }
    stage_direct<BN, BKROW, NT>(rsb, B, b_tile(s % 3), n0, k0, N, kend);
  };

  const int nk = (kend - kbeg + kBK - 1) / kBK;
  if (nk > 0) issue(0);
  if (nk > 1) issue(1);
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) wait_vm<kLoads>();
    else wait_vm<0>();
    lds_barrier();     // stage kt is in LDS; stage kt + 1 may still be loading
    if (kt + 2 < nk) issue(kt + 2);
    const bf16* ta = a_tile(kt % 3);
    const bf16* tb = b_tile(kt % 3);
#pragma unroll
    for (int c = 0; c < kBK / 16; ++c) {
      bf16x8 bo[2];
#pragma unroll
      for (int j = 0; j < 2; ++j)
        bo[j] = BKROW ? row_operand<BN>(tb, 16 * c, wn + 32 * j, lane) : tr_operand<BN>(tb, 16 * c, wn + 32 * j, lane);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bf16x8 ao =
            AKROW ? row_operand<kBM>(ta, 16 * c, wm + 32 * i, lane) : tr_operand<kBM>(ta, 16 * c, wm + 32 * i, lane);
#pragma unroll
        for (int j = 0; j < 2; ++j) mma16(acc[i][j], ao, bo[j]);
      }
    }
  }
  __syncthreads();   // every wave is done with the stages: their LDS now stages the epilogue

  // Epilogue, 32 rows of the wave's block at a time: acc[i][j] holds rows
  // 32i + 8g + 4h + x (register 4g + x), column 32j + lane % 32; they go
  // through the wave's own LDS tile so that each lane then handles 8
  // consecutive columns of one row with 16-byte loads and stores.
  float* et = reinterpret_cast<float*>(smem) + wave * 32 * kEpiS;
  const int h = lane >> 5, col = lane & 31;
  const int er = lane >> 1, ec = (lane & 1) * 32;     // this lane's row and first column when reading back
  constexpr bool kCol = EPI == EPI_GELU_GRAD;
  float cs[kCol ? 4 : 1][8] = {};                      // this lane's column sums over its four rows
  // per-column epilogue constants of this lane's 32 columns, loaded once
  // for the four row blocks (LayerNorm fold: s and c; bias)
  constexpr bool kLn = EPI == EPI_LN_QKV || EPI == EPI_LN_GELU;
  constexpr int kPc = kLn ? 2 : (EPI == EPI_BIAS_RES ? 1 : 0);
  float pc[kPc > 0 ? kPc : 1][4][8];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int n = n0 + wn + ec + 8 * q;     // N is a multiple of 8
#pragma unroll
    for (int a = 0; a < kPc; ++a) {
      const float* src = kLn ? (a == 0 ? ep.lns : ep.lnc) : ep.bias;
      float4 lo = make_float4(0.f, 0.f, 0.f, 0.f), hi = lo;
      if (n < N) {
        lo = *reinterpret_cast<const float4*>(src + n);
        hi = *reinterpret_cast<const float4*>(src + n + 4);
      }
      pc[a][q][0] = lo.x; pc[a][q][1] = lo.y; pc[a][q][2] = lo.z; pc[a][q][3] = lo.w;
      pc[a][q][4] = hi.x; pc[a][q][5] = hi.y; pc[a][q][6] = hi.z; pc[a][q][7] = hi.w;
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) et[(8 * (r / 4) + 4 * h + (r % 4)) * kEpiS + 32 * j + col] = acc[i][j][r];
    __builtin_amdgcn_wave_barrier();
    const int m = m0 + wm + 32 * i + er;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int n = n0 + wn + ec + 8 * q;
      const float4 lo = *reinterpret_cast<const float4*>(et + er * kEpiS + ec + 8 * q);
      const float4 hi = *reinterpret_cast<const float4*>(et + er * kEpiS + ec + 8 * q + 4);
      float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
      if (m >= M || n >= N) continue;
      const int64_t o = (int64_t)m * N + n;
      if (EPI == EPI_LN_QKV || EPI == EPI_LN_GELU) {
        const float mu = ep.mean[m], rs = ep.rstd[m];
        bf16x8 t, g;
#pragma unroll
        for (int x = 0; x < 8; ++x) {
          const float y = rs * (v[x] - mu * pc[0][q][x]) + pc[1][q][x];
          t[x] = (bf16)y;
          if (EPI == EPI_LN_GELU) g[x] = (bf16)gelu_f(y);
        }
        if (EPI == EPI_LN_QKV) {
          const int blk = n / ep.split;
          *reinterpret_cast<bf16x8*>(ep.out[blk] + (int64_t)m * ep.split + (n - blk * ep.split)) = t;
        } else {
          *reinterpret_cast<bf16x8*>(ep.out[0] + o) = t;
          *reinterpret_cast<bf16x8*>(ep.out2 + o) = g;
        }
      } else if (EPI == EPI_BIAS_RES) {
        const bf16x8 res = *reinterpret_cast<const bf16x8*>(ep.aux + o);
        bf16x8 t;
#pragma unroll
        for (int x = 0; x < 8; ++x) t[x] = (bf16)(v[x] + pc[0][q][x] + (float)res[x]);
        *reinterpret_cast<bf16x8*>(ep.out[0] + o) = t;
      } else if (EPI == EPI_GELU_GRAD) {
        const bf16x8 hv = *reinterpret_cast<const bf16x8*>(ep.aux + o);
        bf16x8 t;
#pragma unroll
        for (int x = 0; x < 8; ++x) t[x] = (bf16)(v[x] * gelu_grad_f((float)hv[x]));
        *reinterpret_cast<bf16x8*>(ep.out[0] + o) = t;
        if constexpr (kCol) {
#pragma unroll
          for (int x = 0; x < 8; ++x) cs[q][x] += (float)t[x];
        }
      } else if (EPI == EPI_F32 || EPI == EPI_F32_ACC) {
        float* dst = ep.outf + (EPI == EPI_F32 ? (int64_t)blockIdx.z * M * N : 0) + o;
        if (EPI == EPI_F32_ACC) {
          const float4 a0 = *reinterpret_cast<const float4*>(dst);
          const float4 a1 = *reinterpret_cast<const float4*>(dst + 4);
          v[0] += a0.x; v[1] += a0.y; v[2] += a0.z; v[3] += a0.w;
          v[4] += a1.x; v[5] += a1.y; v[6] += a1.z; v[7] += a1.w;
        }
        *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
        *reinterpret_cast<float4*>(dst + 4) = make_float4(v[4], v[5], v[6], v[7]);
      } else {
        bf16x8 t;
#pragma unroll
        for (int x = 0; x < 8; ++x) t[x] = (bf16)v[x];
        *reinterpret_cast<bf16x8*>(ep.out[0] + o) = t;
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
  if constexpr (kCol) {
    // the wave's 32 lanes of each parity hold four-row sums of the same 32
    // columns: through the wave's staging tile, lane c then adds column c
    // over the 32 lanes' rows in order
    if (ep.colpart != nullptr) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int x = 0; x < 8; ++x) et[er * kEpiS + ec + 8 * q + x] = cs[q][x];
      __builtin_amdgcn_wave_barrier();
      float sum = 0.0f;
      for (int r = 0; r < 32; ++r) sum += et[r * kEpiS + lane];
      const int n = n0 + wn + lane;
      if (n < N) ep.colpart[(int64_t)(2 * tm + wm / 128) * N + n] = sum;
    }
  }
}

// LayerNorm applied to a token matrix (the backward's weight gradients take
// the normalised activations as an operand): out = (z - mean) rstd gamma +
// beta, rounded to bf16; one thread per 8 channels.
__global__ __launch_bounds__(256) void ln_apply_kernel(const bf16* __restrict__ z, const float* __restrict__ mean,
                                                      const float* __restrict__ rstd, const float* __restrict__ gamma,
                                                      const float* __restrict__ beta, bf16* __restrict__ out, int T,
                                                      int C) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int c8 = C / 8;
  if (idx >= (int64_t)T * c8) return;
  const int t = (int)(idx / c8);
  const int c = 8 * (int)(idx - (int64_t)t * c8);
  const bf16x8 v = *reinterpret_cast<const bf16x8*>(z + (int64_t)t * C + c);
  const float mu = mean[t], rs = rstd[t];
  bf16x8 o;
#pragma unroll
  for (int x = 0; x < 8; ++x) o[x] = (bf16)(((float)v[x] - mu) * rs * gamma[c + x] + beta[c + x]);
  *reinterpret_cast<bf16x8*>(out + (int64_t)t * C + c) = o;
}

// LayerNorm folded into the following linear layer: with
// LN(x)_k = (x_k - mean) rstd gamma_k + beta_k,
//   LN(x) W^T + b = rstd (x Wf^T - mean s) + c,
//   Wf[n][k] = bf16(W[n][k] gamma_k),  s_n = sum_k Wf[n][k],
//   c_n = b_n + sum_k W[n][k] beta_k,
// so the GEMM runs on the raw activations and the epilogue normalises.  One
// wave per output row n.
__global__ __launch_bounds__(256) void ln_fold_kernel(const bf16* __restrict__ W, const float* __restrict__ gamma,
                                                     const float* __restrict__ beta, const float* __restrict__ bias,
                                                     bf16* __restrict__ Wf, float* __restrict__ lns,
                                                     float* __restrict__ lnc, int N, int K) {
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (n >= N) return;
  float sacc = 0.0f, cacc = 0.0f;
  for (int k = 8 * lane; k < K; k += 512) {
    const bf16x8 w = *reinterpret_cast<const bf16x8*>(W + (int64_t)n * K + k);
    bf16x8 f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      f[i] = (bf16)((float)w[i] * gamma[k + i]);
      sacc += (float)f[i];
      cacc += (float)w[i] * beta[k + i];
    }
    *reinterpret_cast<bf16x8*>(Wf + (int64_t)n * K + k) = f;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    sacc += __shfl_xor(sacc, o, 64);
    cacc += __shfl_xor(cacc, o, 64);
  }
  if (lane == 0) {
    lns[n] = sacc;
    lnc[n] = cacc + bias[n];
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

// Mean and 1/std of each row, one wave a row: the row is read once into
// registers (C <= 2048: four 8-element chunks a lane) and the variance is
// taken about the mean from there.
__global__ __launch_bounds__(kRowThreads) void ln_stats_kernel(const bf16* __restrict__ x, float* __restrict__ mean,
                                                               float* __restrict__ rstd, int T, int C, float eps) {
  const int row = blockIdx.x * (kRowThreads / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= T) return;
  const bf16* p = x + (int64_t)row * C;
  bf16x8 v[4];
#pragma unroll
  for (int c = 0; c < 4; ++c)
    if (8 * lane + 512 * c < C) v[c] = *reinterpret_cast<const bf16x8*>(p + 8 * lane + 512 * c);
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < 4; ++c)
    if (8 * lane + 512 * c < C)
#pragma unroll
      for (int i = 0; i < 8; ++i) s += (float)v[c][i];
  const float mu = wave_sum(s) / (float)C;
  float q = 0.0f;
#pragma unroll
  for (int c = 0; c < 4; ++c)
    if (8 * lane + 512 * c < C)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float d = (float)v[c][i] - mu;
        q += d * d;
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

// NCH = ceil(C / 512) chunk slots a lane (registers for C, not for 2048)
template <typename DY, int NCH>
__global__ __launch_bounds__(kRowThreads) void ln_bwd_kernel(
    const DY* __restrict__ dy, const bf16* __restrict__ z, const float* __restrict__ mean,
    const float* __restrict__ rstd, const float* __restrict__ gamma, const bf16* __restrict__ dres,
    bf16* __restrict__ dz, float* __restrict__ part, int T, int C, int rows_per_wave) {
  const int gw = blockIdx.x * (kRowThreads / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  float dg[NCH][8], db[NCH][8];
#pragma unroll
  for (int c = 0; c < NCH; ++c)
#pragma unroll
    for (int i = 0; i < 8; ++i) dg[c][i] = db[c][i] = 0.0f;
  const int r0 = gw * rows_per_wave;
  const int r1 = min(T, r0 + rows_per_wave);
  const float invC = 1.0f / (float)C;
  for (int row = r0; row < r1; ++row) {
    const float mu = mean[row], rs = rstd[row];
    float zh[NCH][8], gg[NCH][8];
    float s1 = 0.0f, s2 = 0.0f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int ch = 8 * (lane + 64 * c);
      if (ch < C) {
        const bf16x8 zv = *reinterpret_cast<const bf16x8*>(z + (int64_t)row * C + ch);
        float d[8];
        if constexpr (sizeof(DY) == 4) {
          const float4 d0 = *reinterpret_cast<const float4*>(dy + (int64_t)row * C + ch);
          const float4 d1 = *reinterpret_cast<const float4*>(dy + (int64_t)row * C + ch + 4);
          d[0] = d0.x; d[1] = d0.y; d[2] = d0.z; d[3] = d0.w; d[4] = d1.x; d[5] = d1.y; d[6] = d1.z; d[7] = d1.w;
        } else {
          const bf16x8 dv = *reinterpret_cast<const bf16x8*>(dy + (int64_t)row * C + ch);
#pragma unroll
          for (int i = 0; i < 8; ++i) d[i] = (float)dv[i];
        }
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
    for (int c = 0; c < NCH; ++c) {
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
  for (int c = 0; c < NCH; ++c) {
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

// Column sums of a bf16 matrix, per slice of rows:
// part[s][col] = sum over rows [s * rows_per, (s+1) * rows_per) - the bias
// gradients, reduced afterwards in slice order.  Thread = 8 columns.
__global__ __launch_bounds__(kRowThreads) void colsum_kernel(Mat X, int ncols, float* __restrict__ part,
                                                             int rows_per) {
  const int c8 = blockIdx.x * kRowThreads + threadIdx.x;
  if (8 * c8 >= ncols) return;
  const int s = blockIdx.y;
  const int r0 = s * rows_per, r1 = min(X.rows, r0 + rows_per);
  // a three-part X (segw > 0): column c of part c / segw
  const bf16* xb = X.p;
  int col = 8 * c8;
  if (X.segw > 0) {
    const int sg = col / X.segw;
    xb += sg * X.segstride;
    col -= sg * X.segw;
  }
  auto at = [&](int r) { return reinterpret_cast<const bf16x8*>(xb + (int64_t)r * X.ld + col); };
  // four independent partial sums (rows r, r+1, r+2, r+3 of each step), so
  // that four loads are in flight; combined in a fixed order at the end
  float acc[4][8] = {};
  int r = r0;
  for (; r + 4 <= r1; r += 4) {
    bf16x8 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = *at(r + u);
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[u][i] += (float)v[u][i];
  }
  for (; r < r1; ++r) {
    const bf16x8 v = *at(r);
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[0][i] += (float)v[i];
  }
#pragma unroll
  for (int i = 0; i < 8; ++i)
    part[(int64_t)s * ncols + 8 * c8 + i] = (acc[0][i] + acc[1][i]) + (acc[2][i] + acc[3][i]);
}

// grp[g][i] = sum of part[s][i] over s in [g * per, (g + 1) * per), in
// order (n entries per slice).
__global__ __launch_bounds__(kRowThreads) void group_sum_kernel(const float* __restrict__ part, float* __restrict__ grp,
                                                                int n, int per) {
  const int i = blockIdx.x * kRowThreads + threadIdx.x;
  if (i >= n) return;
  const int g = blockIdx.y;
  float acc = 0.0f;
  for (int sl = g * per; sl < (g + 1) * per; ++sl) acc += part[(int64_t)sl * n + i];
  grp[(int64_t)g * n + i] = acc;
}

// out[i] = sum over s < nslice of part[s * stride + i], in slice order (few
// slices, many outputs: the weight gradients).
__global__ __launch_bounds__(kRowThreads) void slice_sum_kernel(const float* __restrict__ part, float* __restrict__ out,
                                                                int64_t n, int64_t stride, int nslice) {
  const int64_t i = (int64_t)blockIdx.x * kRowThreads + threadIdx.x;
  if (i >= n) return;
  float acc = 0.0f;
  int s = 0;
  for (; s + 8 <= nslice; s += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = part[(int64_t)(s + u) * stride + i];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc += v[u];
  }
  for (; s < nslice; ++s) acc += part[(int64_t)s * stride + i];
  out[i] = acc;
}

// The same for many slices and few outputs (the column sums' 512 row
// slices): a workgroup takes 64 consecutive i; its four waves sum the slices
// s = 4j + wave in order, and the four sums are added in wave order (a fixed
// order for every i), so that the slice list is four short dependent chains.
__global__ __launch_bounds__(256) void slice_sum4_kernel(const float* __restrict__ part, float* __restrict__ out,
                                                        int64_t n, int64_t stride, int nslice) {
  __shared__ float red[4][64];
  const int c = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int64_t i = (int64_t)blockIdx.x * 64 + c;
  float acc = 0.0f;
  if (i < n) {
    int s = q;
    for (; s + 28 < nslice; s += 32) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = part[(int64_t)(s + 4 * u) * stride + i];
#pragma unroll
      for (int u = 0; u < 8; ++u) acc += v[u];
    }
    for (; s < nslice; s += 4) acc += part[(int64_t)s * stride + i];
  }
  red[q][c] = acc;
  __syncthreads();
  if (q == 0 && i < n) out[i] = ((red[0][c] + red[1][c]) + red[2][c]) + red[3][c];
}

// out[c][r] = in[r][c] for a rows x cols bf16 matrix: the backward's copies
// of the weights in [N][K] order, so that its data-gradient products read
// their B operand with straight rather than transposed LDS reads (a few MB,
// once per backward).
__global__ __launch_bounds__(256) void transpose_kernel(const bf16* __restrict__ in, bf16* __restrict__ out,
                                                        int rows, int cols) {
  __shared__ bf16 t[32][33];
  const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int y = ty; y < 32; y += 8) {
    const int r = r0 + y, c = c0 + tx;
    if (r < rows && c < cols) t[y][tx] = in[(int64_t)r * cols + c];
  }
  __syncthreads();
  for (int y = ty; y < 32; y += 8) {
    const int c = c0 + y, r = r0 + tx;
    if (c < cols && r < rows) out[(int64_t)c * rows + r] = t[tx][y];
  }
}

// ---------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------
template <bool AKROW, bool BKROW, int EPI, bool SEG = false, int NW = 8>
static hipError_t gemm(const Mat& A, const Mat& B, const EpiArgs& ep, int M, int N, int K, int nsplit,
                       hipStream_t st) {
  constexpr int BN = NW * 32;
  // three stages: 96 KB (eight waves), 72 KB (four)
  constexpr size_t lds = 3 * (size_t)(kBM + BN) * kBK * sizeof(bf16);
  const int tiles = ((M + kBM - 1) / kBM) * ((N + BN - 1) / BN);
  const int kslice = ((K + nsplit - 1) / nsplit + kBK - 1) / kBK * kBK;
  hipLaunchKernelGGL((gemm_kernel<AKROW, BKROW, EPI, SEG, NW>), dim3(tiles, 1, nsplit), dim3(NW * 64), lds, st, A, B,
                     ep, M, N, K, kslice);
  return hipGetLastError();
}


static Mat mat(const void* p, int ld, int rows) {
  Mat m;
  m.p = (const bf16*)p;
  m.ld = ld;
  m.rows = rows;
  m.segw = 0;
  m.segstride = 0;
  return m;
}

// A product whose 256 x 256 tiles do not fill whole rounds of one
// workgroup per CU (N = C: 3 column tiles by ceil(T / 256) row tiles, 6.3
// rounds on the 128x1080 grid): the rows of the whole rounds go to the
// eight-wave form, the rest to the four-wave form, whose 256 x 128 tiles
// spread the last partial round over twice as many workgroups.  A is
// K-major and the epilogue writes (and, for the residual, reads) rows of
// N, offset by the first part's rows.
template <bool BKROW, int EPI, bool SEG = false>
static hipError_t gemm_rounds(const Mat& A, const Mat& B, const EpiArgs& ep, int M, int N, int K, hipStream_t st) {
  static_assert(EPI == EPI_BF16 || EPI == EPI_BIAS_RES, "row offsets are set for these epilogues");
  const int ntn = (N + kBN - 1) / kBN, nM = (M + kBM - 1) / kBM;
  int r1 = ((nM * ntn) / kMaxCusBlock) * kMaxCusBlock / ntn;   // row tiles in whole rounds
  while (r1 > 0 && (r1 * ntn) % 8 != 0) --r1;   // a tile count the XCD-grouped order takes
  if (r1 == 0 || r1 >= nM) return gemm<true, BKROW, EPI, SEG>(A, B, ep, M, N, K, 1, st);
  const int m1 = r1 * kBM;
  hipError_t e = gemm<true, BKROW, EPI, SEG>(A, B, ep, m1, N, K, 1, st);
  if (e != hipSuccess) return e;
  Mat a2 = A;
  a2.p = A.p + (int64_t)m1 * A.ld;
  a2.rows = A.rows - m1;
  EpiArgs e2 = ep;
  e2.out[0] = ep.out[0] + (int64_t)m1 * N;
  if (EPI == EPI_BIAS_RES) e2.aux = ep.aux + (int64_t)m1 * N;
  return gemm<true, BKROW, EPI, SEG, 4>(a2, B, e2, M - m1, N, K, 1, st);
}


constexpr float kLnEps = 1e-5f;

hipError_t launch_attn_fwd(const Geo& g, int dt, bool nhwc, const void* q, const void* k, const void* v,
                           const float* table, void* o, void* olo, float* lse, hipStream_t st);
hipError_t launch_attn_bwd(const Geo& g, int dt, bool nhwc, const void* q, const void* k, const void* v,
                           const void* o, const void* olo, const void* dout, const float* lse,
                           const float* table, void* dq, void* dk, void* dv, float* dtab, void* ws,
                           hipStream_t st);
size_t bwd_workspace(const Geo& g, int dt);

static hipError_t ln_stats(const void* x, float* mu, float* rs, int T, int C, hipStream_t st) {
  const int per = kRowThreads / 64;
  hipLaunchKernelGGL(ln_stats_kernel, dim3((T + per - 1) / per), dim3(kRowThreads), 0, st, (const bf16*)x, mu, rs,
                     T, C, kLnEps);
  return hipGetLastError();
}

static size_t al(size_t x) { return (x + 255) / 256 * 256; }

// Forward workspace: the folded QKV and fc1 weights and their per-output
// sums and constants.
struct FwdWs {
  size_t wq, wf, sq, cq, sf, cf, total;
};
static FwdWs fwd_ws(const Geo& g) {
  const size_t C = g.C;
  FwdWs w;
  size_t off = 0;
  w.wq = off; off += al(3 * C * C * 2);
  w.wf = off; off += al(4 * C * C * 2);
  w.sq = off; off += al(3 * C * 4);
  w.cq = off; off += al(3 * C * 4);
  w.sf = off; off += al(4 * C * 4);
  w.cf = off; off += al(4 * C * 4);
  w.total = off;
  return w;
}
size_t block_fwd_workspace(const Geo& g) { return fwd_ws(g).total; }

static hipError_t ln_fold(const void* W, const float* gamma, const float* beta, const float* bias, bf16* Wf,
                          float* lns, float* lnc, int N, int K, hipStream_t st) {
  hipLaunchKernelGGL(ln_fold_kernel, dim3((N + 3) / 4), dim3(256), 0, st, (const bf16*)W, gamma, beta, bias, Wf, lns,
                     lnc, N, K);
  return hipGetLastError();
}

hipError_t launch_block_fwd(const Geo& g, const void* x, const BlockParams& p, const float* table, void* x2,
                            const BlockSaved& s, void* wsv, hipStream_t st) {
  const int T = g.B * g.H * g.W, C = g.C;
  const FwdWs w = fwd_ws(g);
  char* ws = reinterpret_cast<char*>(wsv);
  bf16* wq = reinterpret_cast<bf16*>(ws + w.wq);
  bf16* wf = reinterpret_cast<bf16*>(ws + w.wf);
  float *sq = reinterpret_cast<float*>(ws + w.sq), *cq = reinterpret_cast<float*>(ws + w.cq);
  float *sf = reinterpret_cast<float*>(ws + w.sf), *cf = reinterpret_cast<float*>(ws + w.cf);
  hipError_t e;
  EpiArgs ep = {};
#define TERRA_TRY(x)                    \
  do {                                  \
    if ((e = (x)) != hipSuccess) return e; \
  } while (0)
  // LN1 statistics; qkv = LN1(x) W_qkv^T + b_qkv with LN1 folded into the
  // weights and the epilogue, written as Q, K, V (NHWC)
  TERRA_TRY(ln_stats(x, s.mu1, s.rstd1, T, C, st));
  TERRA_TRY(ln_fold(p.w_qkv, p.ln1_g, p.ln1_b, p.b_qkv, wq, sq, cq, 3 * C, C, st));
  ep.out[0] = (bf16*)s.q; ep.out[1] = (bf16*)s.k; ep.out[2] = (bf16*)s.v; ep.split = C;
  ep.mean = s.mu1; ep.rstd = s.rstd1; ep.lns = sq; ep.lnc = cq;
  TERRA_TRY((gemm<true, true, EPI_LN_QKV, false, 4>(mat(x, C, T), mat(wq, C, 3 * C), ep,
                                                                    T, 3 * C, C, 1, st)));
  // windowed attention with the route fused in
  TERRA_TRY(launch_attn_fwd(g, 1, true, s.q, s.k, s.v, table, s.o, nullptr, s.lse, st));
  // x1 = x + o W_p^T + b_p
  ep = EpiArgs{};
  ep.out[0] = (bf16*)s.x1; ep.split = C; ep.aux = (const bf16*)x; ep.bias = p.b_proj;
  TERRA_TRY((gemm<true, true, EPI_BIAS_RES, false, 4>(mat(s.o, C, T), mat(p.w_proj, C, C), ep, T, C, C, 1, st)));
  // h = LN2(x1) W_1^T + b_1 (LN2 folded), a = GELU(h)
  TERRA_TRY(ln_stats(s.x1, s.mu2, s.rstd2, T, C, st));
  TERRA_TRY(ln_fold(p.w_fc1, p.ln2_g, p.ln2_b, p.b_fc1, wf, sf, cf, 4 * C, C, st));
  ep = EpiArgs{};
  ep.out[0] = (bf16*)s.h; ep.split = 4 * C; ep.out2 = (bf16*)s.a;
  ep.mean = s.mu2; ep.rstd = s.rstd2; ep.lns = sf; ep.lnc = cf;
  TERRA_TRY((gemm<true, true, EPI_LN_GELU>(mat(s.x1, C, T), mat(wf, C, 4 * C), ep, T, 4 * C, C, 1, st)));
  // x2 = x1 + a W_2^T + b_2
  ep = EpiArgs{};
  ep.out[0] = (bf16*)x2; ep.split = C; ep.aux = (const bf16*)s.x1; ep.bias = p.b_fc2;
  TERRA_TRY((gemm_rounds<true, EPI_BIAS_RES>(mat(s.a, 4 * C, T), mat(p.w_fc2, 4 * C, C), ep, T, C, 4 * C, st)));
#undef TERRA_TRY
  return hipSuccess;
}

// Token slices of a weight gradient dW[Nl][Kl] over T tokens.
static int wgrad_slices(int T, int Nl, int Kl, int cap) {
  const int tiles = ((Nl + kBM - 1) / kBM) * ((Kl + kBN - 1) / kBN);
  // two whole rounds of one workgroup per CU (a third, nearly empty round
  // would leave most CUs idle for a whole slice)
  int n = (2 * kMaxCusBlock) / tiles;
  const int per = (T + n - 1) / n;
  if (per < 4 * kBK) n = (T + 4 * kBK - 1) / (4 * kBK);  // at least four stages a slice
  return n < 1 ? 1 : (n > cap ? cap : n);
}

// Backward workspace layout (bytes, 256-aligned pieces).
struct BwdWs {
  size_t dh, dln, dx1, dO, dq, dk, dv, ln, wt, attn, wpart, cpart, lpart, total;
  int wsplit, cslices, lnwaves, rows_per_wave, cpart_rows, lgroups;
};

// A pure function of the geometry: the attention part is sized for kMaxCus
// whatever device the call runs on.
static BwdWs block_ws(const Geo& geo) {
  Geo g = geo;
  g.cus = kMaxCus;
  BwdWs w;
  const size_t T = (size_t)g.B * g.H * g.W, C = g.C;
  w.wsplit = 64;                         // most contraction (token) slices of a weight gradient
  w.cslices = 512;                       // row slices of the bias-gradient column sums
  w.cpart_rows = (int)((T + w.cslices - 1) / w.cslices);
  w.lnwaves = 4096;                      // waves of the LayerNorm backward
  w.rows_per_wave = (int)((T + w.lnwaves - 1) / w.lnwaves);
  w.lgroups = 128;                       // first-level groups of the LayerNorm partials (32 waves each)
  size_t off = 0;
  w.dh = off; off += al(T * 4 * C * 2);
  w.dln = off; off += al(T * C * 4);
  w.dx1 = off; off += al(T * C * 2);
  w.dO = off; off += al(T * C * 2);
  w.dq = off; off += al(T * C * 2);
  w.dk = off; off += al(T * C * 2);
  w.dv = off; off += al(T * C * 2);
  w.ln = off; off += al(T * C * 2);
  w.wt = off; off += al(12 * C * C * 2);  // transposed W_fc2, W_fc1, W_proj, W_qkv
  w.attn = off; off += al(bwd_workspace(g, 1));
  size_t wmax = 0;                       // largest slices x output of the block's weight gradients
  for (int i = 0; i < 4; ++i) {
    const int nl = i == 0 ? (int)C : (i == 1 ? 4 * (int)C : (i == 2 ? 3 * (int)C : (int)C));
    const int kl = i == 0 ? 4 * (int)C : (int)C;
    wmax = std::max(wmax, (size_t)wgrad_slices((int)T, nl, kl, w.wsplit) * nl * kl);
  }
  w.wpart = off; off += al(wmax * 4);
  // column-sum partials: the colsum slices, or the dh product's 2 ceil(T/256) rows
  w.cpart = off; off += al((size_t)std::max((size_t)w.cslices, 2 * ((T + kBM - 1) / kBM)) * 4 * C * 4);
  w.lpart = off; off += al((size_t)w.lnwaves * 2 * C * 4 + (size_t)w.lgroups * 2 * C * 4);
  w.total = off;
  return w;
}

size_t block_bwd_workspace(const Geo& g) { return block_ws(g).total; }

static hipError_t slice_sum(const float* part, float* out, int64_t n, int nslice, hipStream_t st,
                            int64_t stride = -1) {
  if (nslice >= 64) {
    hipLaunchKernelGGL(slice_sum4_kernel, dim3((unsigned)((n + 63) / 64)), dim3(256), 0, st, part, out, n,
                       stride < 0 ? n : stride, nslice);
  } else {
    hipLaunchKernelGGL(slice_sum_kernel, dim3((unsigned)((n + kRowThreads - 1) / kRowThreads)), dim3(kRowThreads), 0,
                       st, part, out, n, stride < 0 ? n : stride, nslice);
  }
  return hipGetLastError();
}

// LayerNorm parameter gradients from the per-wave partials
// [wave][dgamma C | dbeta C]: sums over groups of consecutive waves, then
// over the groups, each in order.
static hipError_t ln_param_grads(const float* lpart, float* dgamma, float* dbeta, int C, const BwdWs& w,
                                 hipStream_t st) {
  float* grp = const_cast<float*>(lpart) + (size_t)w.lnwaves * 2 * C;
  const int per = w.lnwaves / w.lgroups;
  hipLaunchKernelGGL(group_sum_kernel, dim3((2 * C + kRowThreads - 1) / kRowThreads, w.lgroups), dim3(kRowThreads),
                     0, st, lpart, grp, 2 * C, per);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if ((e = slice_sum(grp, dgamma, C, w.lgroups, st, 2 * C)) != hipSuccess) return e;
  return slice_sum(grp + C, dbeta, C, w.lgroups, st, 2 * C);
}

static hipError_t colsum(const Mat& X, int ncols, float* part, float* out, const BwdWs& w, hipStream_t st) {
  hipLaunchKernelGGL(colsum_kernel, dim3((ncols / 8 + kRowThreads - 1) / kRowThreads, w.cslices), dim3(kRowThreads),
                     0, st, X, ncols, part, w.cpart_rows);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return slice_sum(part, out, ncols, w.cslices, st);
}

// Weight gradient dW[Nl][Kl] = dY^T Z over all tokens (dY: T x Nl, Z: T x Kl),
// in token slices, reduced in slice order.  LNB: Z = LN(z) applied while
// staging.

static hipError_t wgrad(const Mat& dY, const Mat& Z, int T, int Nl, int Kl, float* dW, char* ws, const BwdWs& w,
                        hipStream_t st) {
  EpiArgs ep = {};
  float* part = reinterpret_cast<float*>(ws + w.wpart);
  ep.outf = part;
  const int ns = wgrad_slices(T, Nl, Kl, w.wsplit);
  hipError_t e = gemm<false, false, EPI_F32>(dY, Z, ep, Nl, Kl, T, ns, st);
  if (e != hipSuccess) return e;
  return slice_sum(part, dW, (int64_t)Nl * Kl, ns, st);
}

// The three-part operand's buffer resource covers 2 segstride + T C
// elements; its byte offsets must stay below 2^31.
static bool seg_fits(int T, int C, int64_t segstride) {
  return (2 * segstride + (int64_t)T * C) * 2 < ((int64_t)1 << 31);
}

// dWqkv[3C][C] = [dQ dK dV]^T Z over all tokens in one product (dy3: the
// three-part T x 3C operand), in token slices reduced in slice order.
static hipError_t wgrad3(const Mat& dy3, const Mat& Z, int T, int C, float* dW, char* ws, const BwdWs& w,
                         hipStream_t st) {
  EpiArgs ep = {};
  float* part = reinterpret_cast<float*>(ws + w.wpart);
  ep.outf = part;
  const int ns = wgrad_slices(T, 3 * C, C, w.wsplit);
  hipError_t e = gemm<false, false, EPI_F32, true>(dy3, Z, ep, 3 * C, C, T, ns, st);
  if (e != hipSuccess) return e;
  return slice_sum(part, dW, (int64_t)3 * C * C, ns, st);
}

// dz = LayerNorm backward of dy (float32 or bf16) + dres, and the per-wave
// gain/shift partials, with the chunk count C needs.
template <typename DY>
static hipError_t ln_bwd(const DY* dy, const void* z, const float* mean, const float* rstd, const float* gamma,
                         const void* dres, void* dz, float* part, int T, int C, const BwdWs& w, hipStream_t st) {
  const dim3 grid(w.lnwaves / 4), block(kRowThreads);
  const bf16* zb = (const bf16*)z;
  const bf16* rb = (const bf16*)dres;
  bf16* ob = (bf16*)dz;
  switch ((C + 511) / 512) {
    case 1: hipLaunchKernelGGL((ln_bwd_kernel<DY, 1>), grid, block, 0, st, dy, zb, mean, rstd, gamma, rb, ob, part, T,
                               C, w.rows_per_wave); break;
    case 2: hipLaunchKernelGGL((ln_bwd_kernel<DY, 2>), grid, block, 0, st, dy, zb, mean, rstd, gamma, rb, ob, part, T,
                               C, w.rows_per_wave); break;
    case 3: hipLaunchKernelGGL((ln_bwd_kernel<DY, 3>), grid, block, 0, st, dy, zb, mean, rstd, gamma, rb, ob, part, T,
                               C, w.rows_per_wave); break;
    default: hipLaunchKernelGGL((ln_bwd_kernel<DY, 4>), grid, block, 0, st, dy, zb, mean, rstd, gamma, rb, ob, part,
                                T, C, w.rows_per_wave); break;
  }
  return hipGetLastError();
}

static hipError_t transpose(const void* in, bf16* out, int rows, int cols, hipStream_t st) {
  hipLaunchKernelGGL(transpose_kernel, dim3((cols + 31) / 32, (rows + 31) / 32), dim3(256), 0, st, (const bf16*)in,
                     out, rows, cols);
  return hipGetLastError();
}

static hipError_t ln_apply(const void* z, const float* mu, const float* rs, const float* gamma, const float* beta,
                           bf16* out, int T, int C, hipStream_t st) {
  const int64_t n = (int64_t)T * (C / 8);
  hipLaunchKernelGGL(ln_apply_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, (const bf16*)z, mu, rs,
                     gamma, beta, out, T, C);
  return hipGetLastError();
}

hipError_t launch_block_bwd(const Geo& g, const void* dx2, const void* x, const BlockParams& p, const float* table,
                            const BlockSaved& s, void* dx, const BlockGrads& gr, float* dtable, void* wsv,
                            hipStream_t st) {
  const int T = g.B * g.H * g.W, C = g.C;
  const BwdWs w = block_ws(g);
  char* ws = reinterpret_cast<char*>(wsv);
  bf16* dh = reinterpret_cast<bf16*>(ws + w.dh);
  float* dln = reinterpret_cast<float*>(ws + w.dln);
  bf16* dlnb = reinterpret_cast<bf16*>(ws + w.dln);     // the same buffer holding bf16
  bf16* dx1 = reinterpret_cast<bf16*>(ws + w.dx1);
  bf16* dO = reinterpret_cast<bf16*>(ws + w.dO);
  bf16* dqkv[3] = {reinterpret_cast<bf16*>(ws + w.dq), reinterpret_cast<bf16*>(ws + w.dk),
                   reinterpret_cast<bf16*>(ws + w.dv)};
  float* cpart = reinterpret_cast<float*>(ws + w.cpart);
  float* lpart = reinterpret_cast<float*>(ws + w.lpart);
  bf16* lnb = reinterpret_cast<bf16*>(ws + w.ln);
  hipError_t e;
  EpiArgs ep = {};
#define TERRA_TRY(x)                    \
  do {                                  \
    if ((e = (x)) != hipSuccess) return e; \
  } while (0)
  // the weights in [N][K] order for the data-gradient products
  bf16* wt_fc2 = reinterpret_cast<bf16*>(ws + w.wt);        // [4C][C]
  bf16* wt_fc1 = wt_fc2 + (size_t)4 * C * C;                // [C][4C]
  bf16* wt_proj = wt_fc1 + (size_t)4 * C * C;               // [C][C]
  bf16* wt_qkv = wt_proj + (size_t)C * C;                   // [C][3C]
  TERRA_TRY(transpose(p.w_fc2, wt_fc2, C, 4 * C, st));
  TERRA_TRY(transpose(p.w_fc1, wt_fc1, 4 * C, C, st));
  TERRA_TRY(transpose(p.w_proj, wt_proj, C, C, st));
  TERRA_TRY(transpose(p.w_qkv, wt_qkv, 3 * C, C, st));
  // x2 = x1 + a W2^T + b2:  dW2 = dx2^T a, db2 = colsum(dx2), dh = (dx2 W2) * GELU'(h)
  TERRA_TRY(wgrad(mat(dx2, C, T), mat(s.a, 4 * C, T), T, C, 4 * C, gr.w_fc2, ws, w, st));
  TERRA_TRY(colsum(mat(dx2, C, T), C, cpart, gr.b_fc2, w, st));
  // db1 = colsum(dh) from the same epilogue: per-wave partial rows, then a
  // fixed-order sum of the 2 ceil(T / 256) partials
  ep.out[0] = dh; ep.split = 4 * C; ep.aux = (const bf16*)s.h; ep.colpart = cpart;
  TERRA_TRY((gemm<true, true, EPI_GELU_GRAD, false, 4>(mat(dx2, C, T), mat(wt_fc2, C, 4 * C), ep, T, 4 * C, C, 1, st)));
  TERRA_TRY(slice_sum(cpart, gr.b_fc1, 4 * C, 2 * ((T + kBM - 1) / kBM), st));
  // h = LN2(x1) W1^T + b1:  dW1 = dh^T LN2(x1), db1 = colsum(dh), dln2 = dh W1
  TERRA_TRY(ln_apply(s.x1, s.mu2, s.rstd2, p.ln2_g, p.ln2_b, lnb, T, C, st));
  TERRA_TRY(wgrad(mat(dh, 4 * C, T), mat(lnb, C, T), T, 4 * C, C, gr.w_fc1, ws, w, st));
  // dln2 in bf16, like the other gradients the products hand on
  ep = EpiArgs{};
  ep.out[0] = dlnb; ep.split = C;
  TERRA_TRY((gemm_rounds<true, EPI_BF16>(mat(dh, 4 * C, T), mat(wt_fc1, 4 * C, C), ep, T, C, 4 * C, st)));
  // dx1 = dx2 + LN2 backward
  TERRA_TRY(ln_bwd(dlnb, s.x1, s.mu2, s.rstd2, p.ln2_g, dx2, dx1, lpart, T, C, w, st));
  TERRA_TRY(ln_param_grads(lpart, gr.ln2_g, gr.ln2_b, C, w, st));
  // x1 = x + o Wp^T + bp:  dWp = dx1^T o, dbp = colsum(dx1), dO = dx1 Wp
  TERRA_TRY(wgrad(mat(dx1, C, T), mat(s.o, C, T), T, C, C, gr.w_proj, ws, w, st));
  TERRA_TRY(colsum(mat(dx1, C, T), C, cpart, gr.b_proj, w, st));
  ep = EpiArgs{};
  ep.out[0] = dO; ep.split = C;
  TERRA_TRY((gemm<true, true, EPI_BF16, false, 4>(mat(dx1, C, T), mat(wt_proj, C, C), ep, T, C, C, 1, st)));
  // attention backward (route fused in)
  TERRA_TRY(launch_attn_bwd(g, 1, true, s.q, s.k, s.v, s.o, nullptr, dO, s.lse, table, dqkv[0], dqkv[1],
                            dqkv[2], dtable, ws + w.attn, st));
  // qkv = LN1(x) Wqkv^T + bqkv, one third (Q, K, V) at a time: rows
  // [iC, (i+1)C) of dWqkv = dY_i^T LN1(x), of dbqkv = colsum(dY_i), and
  // dln1 = sum_i dY_i Wqkv[iC:(i+1)C]
  TERRA_TRY(ln_apply(x, s.mu1, s.rstd1, p.ln1_g, p.ln1_b, lnb, T, C, st));
  // dQ, dK, dV sit at equal strides in the workspace: one T x 3C operand of
  // three parts, so that dWqkv is one product over all tokens and dln one
  // product over 3C (instead of three, two of them adding float32 results)
  Mat dy3 = mat(dqkv[0], C, T);
  dy3.segw = C;
  dy3.segstride = (int64_t)(w.dk - w.dq) / 2;
  const bool seg_w = C % kBM == 0 && seg_fits(T, C, dy3.segstride);
  const bool seg_d = C % kBK == 0 && seg_fits(T, C, dy3.segstride);
  if (seg_w) {
    TERRA_TRY(wgrad3(dy3, mat(lnb, C, T), T, C, gr.w_qkv, ws, w, st));
  }
  if (!seg_w) {
    for (int i = 0; i < 3; ++i)
      TERRA_TRY(wgrad(mat(dqkv[i], C, T), mat(lnb, C, T), T, C, C, gr.w_qkv + (size_t)i * C * C, ws, w, st));
  }
  TERRA_TRY(colsum(dy3, 3 * C, cpart, gr.b_qkv, w, st));
  ep = EpiArgs{};
  if (seg_d) {
    ep.out[0] = dlnb; ep.split = C;
    TERRA_TRY((gemm_rounds<true, EPI_BF16, true>(dy3, mat(wt_qkv, 3 * C, C), ep, T, C, 3 * C, st)));
  } else {
    ep.outf = dln;
    for (int i = 0; i < 3; ++i) {
      const bf16* wi = reinterpret_cast<const bf16*>(p.w_qkv) + (size_t)i * C * C;
      if (i == 0) {
        TERRA_TRY((gemm<true, false, EPI_F32>(mat(dqkv[i], C, T), mat(wi, C, C), ep, T, C, C, 1, st)));
      } else {
        TERRA_TRY((gemm<true, false, EPI_F32_ACC>(mat(dqkv[i], C, T), mat(wi, C, C), ep, T, C, C, 1, st)));
      }
    }
  }
  // dx = dx1 + LN1 backward
  if (seg_d) {
    TERRA_TRY(ln_bwd(dlnb, x, s.mu1, s.rstd1, p.ln1_g, dx1, dx, lpart, T, C, w, st));
  } else {
    TERRA_TRY(ln_bwd(dln, x, s.mu1, s.rstd1, p.ln1_g, dx1, dx, lpart, T, C, w, st));
  }
  TERRA_TRY(ln_param_grads(lpart, gr.ln1_g, gr.ln1_b, C, w, st));
#undef TERRA_TRY
  return hipSuccess;
}

}  // namespace terra
