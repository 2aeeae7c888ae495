// Dense projections of the verification step (QKV, O, gate/up, down, LM head).
//
// bf16 path: both operands are pre-packed into 32x16 fragments (lane order of gfx950's
// v_mfma_f32_32x32x16_bf16), so each wave-level load of a fragment is one contiguous
// 1 KiB read.  A workgroup of four waves stages KS fragments of K per step through
// double-buffered LDS and accumulates in fp32.  Small-M (the verify step's
// sum(gamma+1) rows) shapes are HBM-bound on the weight stream; K is split across
// workgroups when there are too few output tiles to fill the 256 CUs, and the fp32
// partial sums are added in a fixed order by the consuming epilogue kernel.
#include "common.h"
#include "kernels.h"

namespace wisp {

template <int WM, int WN, int MT, int NT, int KS>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(const uint16_t *__restrict__ A,
                                                        const uint16_t *__restrict__ W,
                                                        float *__restrict__ C, int M, int N, int K,
                                                        int ldc, int kf_per_split) {
  constexpr int BMF = WM * MT;        // 32-row fragments of A per tile
  constexpr int BNF = WN * NT;        // 32-row fragments of W per tile
  constexpr int A_FR = BMF * KS;
  constexpr int FR = (BMF + BNF) * KS;
  constexpr int PER_T = FR * 64 / 256;
  static_assert((FR * 64) % 256 == 0, "stage must split evenly over 256 threads");
  __shared__ uint4 lds[2][FR][64];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int KF = K >> 4;
  const int kf0 = blockIdx.z * kf_per_split;
  const int kf1 = min(KF, kf0 + kf_per_split);
  const int nstage = (kf1 - kf0 + KS - 1) / KS;
  const int rb0 = blockIdx.y * BMF, nb0 = blockIdx.x * BNF;
  const int MF = (M + 31) >> 5, NF = N >> 5;

  floatx16 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  uint4 pre[PER_T];
  auto load_stage = [&](int st) {
    const int kfs = kf0 + st * KS;
#pragma unroll
    for (int t = 0; t < PER_T; ++t) {
      const int c = tid + 256 * t;
      const int f = c >> 6, lc = c & 63;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (f < A_FR) {
        const int r = rb0 + f / KS, kf = kfs + f % KS;
        if (r < MF && kf < kf1)
          v = *reinterpret_cast<const uint4 *>(A + (((int64_t)r * KF + kf) * 64 + lc) * 8);
      } else {
        const int g = f - A_FR;
        const int n = nb0 + g / KS, kf = kfs + g % KS;
        if (n < NF && kf < kf1)
          v = *reinterpret_cast<const uint4 *>(W + (((int64_t)n * KF + kf) * 64 + lc) * 8);
      }
      pre[t] = v;
    }
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int t = 0; t < PER_T; ++t) {
      const int c = tid + 256 * t;
      lds[buf][c >> 6][c & 63] = pre[t];
    }
  };

  if (nstage > 0) {
    load_stage(0);
    store_stage(0);
  }
  __syncthreads();
  for (int st = 0; st < nstage; ++st) {
    const int buf = st & 1;
    if (st + 1 < nstage) load_stage(st + 1);
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      bf16x8_t a[MT], b[NT];
#pragma unroll
      for (int i = 0; i < MT; ++i) a[i] = as_bf16x8(lds[buf][(wm * MT + i) * KS + kk][lane]);
#pragma unroll
      for (int j = 0; j < NT; ++j) b[j] = as_bf16x8(lds[buf][A_FR + (wn * NT + j) * KS + kk][lane]);
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (st + 1 < nstage) store_stage(buf ^ 1);
    __syncthreads();
  }

  float *Cz = C + (int64_t)blockIdx.z * M * ldc;
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    const int rbase = (rb0 + wm * MT + i) * 32 + 4 * (lane >> 5);
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const int col = (nb0 + wn * NT + j) * 32 + (lane & 31);
      if (col >= N) continue;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = rbase + 8 * (e >> 2) + (e & 3);
        if (row < M) Cz[(int64_t)row * ldc + col] = acc[i][j][e];
      }
    }
  }
}

static constexpr int kKS = 4;

GemmCfg gemm_bf16_plan(int M, int N, int K) {
  GemmCfg c;
  const int mf = (M + 31) / 32;
  int mt = mf <= 2 ? 1 : mf <= 4 ? 2 : mf <= 6 ? 3 : 4;
  c.bm = 2 * mt * 32;
  c.bn = 128;
  const int tiles = ((N + c.bn - 1) / c.bn) * ((M + c.bm - 1) / c.bm);
  const int KF = K / 16;
  int splits = 1;
  if (tiles < 200) {
    splits = (240 + tiles - 1) / tiles;
    const int max_split = KF / (kKS * 4) > 0 ? KF / (kKS * 4) : 1;   // >= 4 stages each
    if (splits > max_split) splits = max_split;
    if (splits > 16) splits = 16;
    if (splits < 1) splits = 1;
  }
  int kps = (KF + splits - 1) / splits;
  kps = (kps + kKS - 1) / kKS * kKS;
  splits = (KF + kps - 1) / kps;
  c.splits = splits;
  c.kf_per_split = kps;
  return c;
}

void gemm_bf16(const uint16_t *A, const uint16_t *W, float *C, int M, int N, int K, int ldc,
               const GemmCfg &cfg, hipStream_t s) {
  dim3 grid((N + cfg.bn - 1) / cfg.bn, (M + cfg.bm - 1) / cfg.bm, cfg.splits);
  switch (cfg.bm) {
    case 64:
      gemm_bf16_kernel<2, 2, 1, 2, kKS><<<grid, 256, 0, s>>>(A, W, C, M, N, K, ldc, cfg.kf_per_split);
      break;
    case 128:
      gemm_bf16_kernel<2, 2, 2, 2, kKS><<<grid, 256, 0, s>>>(A, W, C, M, N, K, ldc, cfg.kf_per_split);
      break;
    case 192:
      gemm_bf16_kernel<2, 2, 3, 2, kKS><<<grid, 256, 0, s>>>(A, W, C, M, N, K, ldc, cfg.kf_per_split);
      break;
    default:
      gemm_bf16_kernel<2, 2, 4, 2, kKS><<<grid, 256, 0, s>>>(A, W, C, M, N, K, ldc, cfg.kf_per_split);
      break;
  }
}

// ---------------------------------------------------------------------------------------
// fp32 path (small models): plain LDS-tiled VALU GEMM, natural row-major operands
// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float *__restrict__ A,
                                                       const float *__restrict__ W,
                                                       float *__restrict__ C, int M, int N, int K,
                                                       int ldc) {
  constexpr int BM = 32, BN = 64, BK = 16;
  __shared__ float As[BK][BM + 1];
  __shared__ float Ws[BK][BN + 1];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  float acc[2][4] = {};
  for (int k0 = 0; k0 < K; k0 += BK) {
    for (int i = tid; i < BM * BK; i += 256) {
      const int r = i / BK, k = i % BK;
      As[k][r] = (m0 + r < M && k0 + k < K) ? A[(int64_t)(m0 + r) * K + k0 + k] : 0.f;
    }
    for (int i = tid; i < BN * BK; i += 256) {
      const int n = i / BK, k = i % BK;
      Ws[k][n] = (n0 + n < N && k0 + k < K) ? W[(int64_t)(n0 + n) * K + k0 + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < BK; ++k)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += As[k][ty * 2 + i] * Ws[k][tx * 4 + j];
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = m0 + ty * 2 + i, c = n0 + tx * 4 + j;
      if (r < M && c < N) C[(int64_t)r * ldc + c] = acc[i][j];
    }
}

void gemm_f32(const float *A, const float *W, float *C, int M, int N, int K, int ldc, hipStream_t s) {
  dim3 grid((N + 63) / 64, (M + 31) / 32, 1);
  gemm_f32_kernel<<<grid, 256, 0, s>>>(A, W, C, M, N, K, ldc);
}

// ---------------------------------------------------------------------------------------
// weight packing: natural [rows][cols] -> 32x16 fragments
// ---------------------------------------------------------------------------------------
__global__ void pack_bf16_kernel(uint16_t *__restrict__ dst, const uint16_t *__restrict__ src,
                                 int rows, int cols) {
  // one thread per (row, 8-column chunk): 16 contiguous bytes in, 16 contiguous bytes out
  const int64_t chunks = (int64_t)rows * (cols / 8);
  for (int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; c < chunks;
       c += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = c / (cols / 8), k = (c % (cols / 8)) * 8;
    const uint4 v = *reinterpret_cast<const uint4 *>(src + r * cols + k);
    *reinterpret_cast<uint4 *>(dst + packed_off(r, k, cols)) = v;
  }
}

void pack_linear_bf16(uint16_t *dst, const uint16_t *src, int rows, int cols, hipStream_t s) {
  const int64_t chunks = (int64_t)rows * (cols / 8);
  int blocks = (int)((chunks + 255) / 256);
  if (blocks > 65535) blocks = 65535;
  pack_bf16_kernel<<<blocks, 256, 0, s>>>(dst, src, rows, cols);
}

}  // namespace wisp
