// Dense projections of the verification step (QKV, O, gate/up, down, LM head).
//
// bf16 path: both operands are pre-packed into 32x16 fragments (lane order of gfx950's
// v_mfma_f32_32x32x16_bf16), so each wave-level load of a fragment is one contiguous
// 1 KiB read.  Every workgroup holds the activations of a block of at most 256 rows
// (staged through double-buffered LDS) while each wave streams its own weight fragments
// straight into a register ring, accumulating in fp32.  The verify step's sum(gamma+1)
// rows make these shapes HBM-bound on the weight stream up to about 315 rows; K is split
// across workgroups when there are too few output tiles to fill the 256 CUs, and the
// fp32 partial sums are added in a fixed order by the consuming epilogue kernel.
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace wisp {

// ---------------------------------------------------------------------------------------
// Weight-streaming variant for the step's small M: each wave keeps a ring of R weight
// fragments in flight (registers, static ring indices, so every wait is exact), consuming
// fragment k and immediately issuing the load of fragment k + R.  Activations are staged
// through double-buffered LDS in chunks of R 16-wide K steps.  Sized for two waves per
// SIMD, i.e. 8 waves x R x NT KiB of weights in flight per CU.
// Every workgroup reads the same activation matrix; to keep concurrent workgroups from
// requesting the same cache lines at once (which serialises on a few L2 channels), each
// workgroup walks its K chunks in a rotated order.  The order is fixed per output tile,
// so results stay deterministic.
// ---------------------------------------------------------------------------------------
template <int WM, int WN, int MT, int NT, int R, int AD>
__global__ __launch_bounds__(64 * WM * WN) void gemm_ring_kernel(const uint16_t *__restrict__ A,
                                                           const uint16_t *__restrict__ W,
                                                           float *__restrict__ C, int M, int N, int K,
                                                           int ldc, int kf_per_split, RowMaxOut rmax) {
  constexpr int BMF = WM * MT;
  constexpr int NTH = 64 * WM * WN;             // threads per workgroup
  constexpr int A_FR = BMF * R;                 // A fragments per chunk
  constexpr int A_PER_T = (A_FR * 64 + NTH - 1) / NTH;
  __shared__ uint4 lds[2][A_FR][64];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int KF = K >> 4, NF = N >> 5;
  const int MF = (M + 31) >> 5;
  // a 1-D grid of (output tile, K split) pairs.  Workgroups are dealt to the 8 XCDs in
  // turn (linear id mod 8), so taking the split from the low digits of the id keeps each
  // split's workgroups on as few XCDs as possible: every XCD's L2 then fetches only the
  // activation columns of its own K ranges instead of all of them
  const int splits = (KF + kf_per_split - 1) / kf_per_split;
  const int zs = (int)(blockIdx.x % (unsigned)splits);
  const int tile = (int)(blockIdx.x / (unsigned)splits);
  const int kf0 = zs * kf_per_split;
  const int kf1 = min(KF, kf0 + kf_per_split);
  // AD = 2: an even number of chunks (a chunk past the split reads zeroed activations)
  const int nch = AD == 2 ? 2 * ((kf1 - kf0 + 2 * R - 1) / (2 * R)) : (kf1 - kf0 + R - 1) / R;
  const int rb0 = blockIdx.y * BMF;
  const int nbw = (tile * WN + wn) * NT;   // this wave's first weight fragment
  const int rot = (int)(((unsigned)tile * 7u + blockIdx.y * 3u) % (unsigned)nch);
  auto chunk_k = [&](int ch) {   // first K step of the ch-th chunk in this workgroup's order;
    return kf0 + ((ch + rot) % nch) * R;   // indices past the end wrap (loads never used)
  };

  floatx16 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // weight fragment (nb, kf) from a clamped address and never masked: K steps outside the
  // split meet zeroed activations (0 x finite weight = 0) and columns beyond N are never
  // stored, so no select has to wait for the load
  auto wload = [&](int j, int kf) {
    const int nb = min(nbw + j, NF - 1);
    const int kq = min(kf, kf1 - 1);
    return ld16_stream(W + (((int64_t)nb * KF + kq) * 64 + lane) * 8);
  };
  uint4 ring[R][NT];
  // first R weight fragments; issued after the first activation chunk's loads, so that
  // the chunk's LDS store (which waits for its loads, and memory counters complete in
  // order) does not also wait for the weights' longer trip from HBM
  auto ring_fill = [&]() {
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int j = 0; j < NT; ++j) ring[r][j] = wload(j, chunk_k(0) + r);
  };

  // Activations reach LDS through register sets.  AD = 2: two sets, chunk c is loaded into
  // set c % 2 two chunks before it is needed and written to LDS buffer c % 2 at the end of
  // chunk c - 1, so an L2 round trip has two chunks of products to hide behind (measured
  // better for the 64-column tiles, whose chunks are short).  AD = 1: one set, each chunk
  // loaded one chunk ahead (measured better for the 32-column tiles).
  static_assert(AD == 1 || AD == 2, "activation prefetch depth");
  uint4 apre[AD][A_PER_T];
  auto aload = [&](int set, int ch) {
#pragma unroll
    for (int t = 0; t < A_PER_T; ++t) {
      const int c = tid + NTH * t;
      const int f = min(c >> 6, A_FR - 1), lc = c & 63;
      const int r = rb0 + f / R, kf = chunk_k(ch) + f % R;
      const bool ok = r < MF && kf < kf1;
      apre[set][t] = keep_if(ok, ld16(A + (((int64_t)(ok ? r : 0) * KF + (ok ? kf : 0)) * 64 + lc) * 8));
    }
  };
  auto astore = [&](int set, int buf) {
#pragma unroll
    for (int t = 0; t < A_PER_T; ++t) {
      const int c = tid + NTH * t;
      if (c < A_FR * 64) lds[buf][c >> 6][c & 63] = apre[set][t];
    }
  };
  // one chunk of R K steps from LDS buffer `buf`, refilling the ring from chunk ch + 1
  // `refill` is false for the last chunk: its refills would fetch fragments that are never
  // used, and the workgroup could not finish before they had arrived
  auto chunk = [&](int buf, int ch, auto refill) {
    constexpr bool kRefill = decltype(refill)::value;
    const int kn = chunk_k(ch + 1);
    uint4 acur[MT], anext[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) acur[i] = lds[buf][(wm * MT + i) * R][lane];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      // activations of step r+1 are read from LDS while step r's products run (the
      // barrier keeps the reads ahead of the products, in registers of their own, so the
      // LDS latency is never exposed)
      if (r + 1 < R) {
#pragma unroll
        for (int i = 0; i < MT; ++i) anext[i] = lds[buf][(wm * MT + i) * R + r + 1][lane];
      }
      __builtin_amdgcn_sched_barrier(0);
      // consume ring slot r, then refill it: the slot's register is dead once the
      // products have issued, so no copy (and no early wait) is needed
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(acur[i]), as_bf16x8(ring[r][j]),
                                                             acc[i][j], 0, 0, 0);
      if constexpr (kRefill) {
#pragma unroll
        for (int j = 0; j < NT; ++j) ring[r][j] = wload(j, kn + r);
      }
      if (r + 1 < R) {
#pragma unroll
        for (int i = 0; i < MT; ++i) acur[i] = anext[i];
      }
      __builtin_amdgcn_sched_barrier(0);   // keep each refill right after its slot's use
    }
  };

  if constexpr (AD == 2) {
    aload(0, 0);
    ring_fill();
    astore(0, 0);
    __syncthreads();
    aload(1, 1);
    aload(0, 2);
    const std::true_type more;
    for (int ch = 0; ch + 2 < nch; ch += 2) {   // straight-line body: every load unconditional
      chunk(0, ch, more);
      astore(1, 1);       // chunk ch + 1
      __syncthreads();
      aload(1, ch + 3);
      chunk(1, ch + 1, more);
      astore(0, 0);       // chunk ch + 2
      __syncthreads();
      aload(0, ch + 4);
    }
    chunk(0, nch - 2, more);   // the last pair (nch is even and >= 2)
    astore(1, 1);
    __syncthreads();
    chunk(1, nch - 1, std::false_type{});
  } else {
    aload(0, 0);
    ring_fill();
    astore(0, 0);
    __syncthreads();
    if (nch > 1) aload(0, 1);
    for (int ch = 0; ch + 1 < nch; ++ch) {
      const int buf = ch & 1;
      chunk(buf, ch, std::true_type{});
      astore(0, buf ^ 1);
      __syncthreads();
      if (ch + 2 < nch) aload(0, ch + 2);
    }
    chunk((nch - 1) & 1, nch - 1, std::false_type{});
  }

  float *Cz = C + (int64_t)zs * M * ldc;
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    const int rbase = (rb0 + wm * MT + i) * 32 + 4 * (lane >> 5);
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      if (nbw + j >= NF) continue;
      const int col = (nbw + j) * 32 + (lane & 31);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = rbase + 8 * (e >> 2) + (e & 3);
        if (row < M) Cz[(int64_t)row * ldc + col] = acc[i][j][e];
      }
    }
  }
  if (rmax.m) {   // LM head (one K range): the row maxima of this tile's columns
    __syncthreads();   // the activation buffers are free now
    tile_row_max<WM, WN, MT, NT>(acc, reinterpret_cast<float *>(&lds[0][0][0]), nbw, NF, N, M,
                                 rb0 * 32, wm * MT, wn, tile, rmax);
  }
}

static constexpr int kNarrowAD = 1;   // activation prefetch depth of the 32-column ring
// From this many 32-row fragments on, the 32-column ring runs 8 waves per workgroup (two per
// SIMD, each on half of the rows), so one wave's products issue while the other waits for
// memory; below it the extra zero rows and doubled weight requests cost more than that buys
static constexpr int kPairedWavesMinMT = 5;

// Launch plan.  LDS-staged output tiles (gemm_tile.hip) for most shapes, the weight ring
// (above) where it streams faster or K does not fit the tile's chunk.  Tile variant by
// row fragments, measured with cold weights on the 8B and 70B projections at 7-1237 rows:
//   1 (<= 32 rows): the 32 x 256 tile with up to 16 K splits for projections of >= 20M
//     weights (at 7 rows QKV 13.4 -> 11.5 us, down 24.0 -> 20.1, LM head 169.5 -> 158.9);
//     the output projection streams as fast on the ring; outputs of 16384-32768 columns
//     (the 8B gate/up) take 64 x 128 tiles in one K range, which fill as many CUs as the
//     32-row tile with two (at 7-23 rows 36-39 us against 38-40) and keep the SwiGLU
//     epilogue (8B steps at B = 1, 2, 4: 4.05 -> 3.84, 4.12 -> 3.90, 4.38 -> 4.12 ms);
//   2: 64 x 128 tiles, 3-4: 128 x 128 (10-23 % faster than the ring on QKV, O, gate/up
//     and down); the LM head stays on the ring (the tiles 7-44 % slower for it at 41-150
//     rows);
//   5: the 192-row tile (QKV 22.1 -> 19.5 us, down 38.4 -> 32.4; gate/up in one K range
//     as fast as the ring with two, 59.0 against 60.5 us, and with the SwiGLU epilogue:
//     8B steps at B = 26 / 28 6.89 / 6.93 -> 6.74 / 6.79 ms);
//     the ring for the LM head;
//   6: 192-row tiles, 256 columns wide only for the LM head (measured over whole steps: for
//     gate/up the 128-column tile in one K range, with the SwiGLU epilogue, beats the
//     256-column one, which needs two K ranges to fill the CUs);
//   7-8: one 256-row tile, 256 columns wide for the LM head (at 240 rows 374 -> 325 us);
//     at 128 columns for the rest (gate/up keeps one K range and its SwiGLU epilogue);
//   9-12: one 384-row tile (at 343-370 rows 10-25 % faster than two 256-row tiles);
//   beyond (> 384 rows): 256 x 256 tiles with the K split below (at 476-1237 rows 9-30 %
//     off QKV + O + down per layer against 384- or 256-row tiles of 128 columns: 8B at
//     1237 rows 371 -> 259 us, 70B at 476 rows 512 -> 380 us; in the 8B step at 1237 rows
//     the projections 21.9 -> 19.3 ms, the row kernels reading the added partials
//     1.87 -> 2.61 ms, the step 45.5 -> 44.2 ms).
// K is split into as many ranges as the work items fit one round of 256 workgroups (at
// most 8, 16 for the 32-row tile), each range keeping at least 8 chunks: not only powers
// of two, since a round that leaves CUs idle costs the GEMM more than the row kernels save
// on fewer partials (QKV of 80 tiles on 3 ranges: 70B at 370 rows 92 -> 72 us alone, the
// 70B step 76.9 -> 75.8 ms; QKV of 48 tiles on 5: 8B at 100 rows 16.5 -> 14.9 us alone, the
// 8B step at 171 rows unchanged, the extra partial costing the row kernels what it saves).
// The ring holds all rows of a row block of at most 256 rows: 64-column wave tiles for
// wide outputs, 32-column tiles with a deeper ring otherwise (8 waves per workgroup from
// kPairedWavesMinMT row fragments on); K split for one resident round.
GemmCfg gemm_bf16_plan(int M, int N, int K) {
  GemmCfg c{};
  const int mf = (M + 31) / 32;
  const int KF = K / 16;
  const bool lm_wide = N >= 65536;
  int variant;
  if (mf == 1) variant = N >= 16384 && N <= 32768 ? 6 : (int64_t)N * K >= ((int64_t)20 << 20) ? 5 : 0;
  else if (mf == 2) variant = lm_wide ? 0 : 6;
  else if (mf <= 4) variant = lm_wide ? 0 : 7;
  else if (mf == 5) variant = lm_wide ? 0 : 1;
  else if (mf == 6) variant = lm_wide ? 4 : 1;
  else if (mf <= 8) variant = lm_wide ? 17 : 13;
  else if (mf <= 12) variant = 12;
  else variant = 17;
  if (variant) {
    const TileShape ts = tile_shape(variant);
    if (K % (16 * ts.ks) == 0) {
      const int tiles = ((mf * 32 + ts.bm - 1) / ts.bm) * ((N + ts.bn - 1) / ts.bn);
      const int KC = K / (16 * ts.ks);
      const int s_max = variant == 5 ? 16 : 8;
      int s = std::max(1, std::min(s_max, 256 / tiles));
      while (s > 1 && KC / s < 8) --s;
      const int kcs = (KC + s - 1) / s;
      c.kind = 4;
      c.variant = variant;
      c.bm = ts.bm;
      c.bn = ts.bn;
      c.mt = ts.bm / 32;
      c.rb = (mf * 32 + ts.bm - 1) / ts.bm;
      c.splits = (KC + kcs - 1) / kcs;
      c.kf_per_split = kcs * ts.ks;
      return c;
    }
  }
  // rows in rb blocks of at most 8 fragments, balanced; each block is one grid row of
  // workgroups that stream the same weights (the grid width is a multiple of 8 for every
  // projection here, so a tile's row blocks share an XCD and its L2)
  c.rb = (mf + 7) / 8;
  int mt = (mf + c.rb - 1) / c.rb;
  c.kind = N >= 16384 ? 2 : (mt >= kPairedWavesMinMT ? 3 : 1);
  if (c.kind == 3 && c.rb > 1) mt += mt & 1;   // paired halves: a block is 2 * ceil(mt / 2) fragments
  c.mt = mt;
  c.bm = 32 * mt;
  c.bn = c.kind == 2 ? 256 : 128;
  const int R = c.kind == 2 ? 4 : 8;
  const int tiles = ((N + c.bn - 1) / c.bn) * c.rb;
  // workgroups resident at once: the ring kernels hold one workgroup per CU (LDS and
  // registers), so more than one round of 256 would leave a partial second round
  const int max_wg = 256;
  int splits = 1;
  while (splits < 16 && tiles * splits * 2 <= max_wg && KF / (splits * 2) >= 4 * R) splits *= 2;
  int kps = (KF + splits - 1) / splits;
  kps = (kps + R - 1) / R * R;
  c.splits = (KF + kps - 1) / kps;
  c.kf_per_split = kps;
  return c;
}

// 32-column ring, 8 waves: two row halves of ceil(mt / 2) fragments each
static void launch_ring_paired(int mt, dim3 grid, const uint16_t *A, const uint16_t *W, float *C, int M,
                               int N, int K, int ldc, int kps, RowMaxOut rm, hipStream_t s) {
  switch ((mt + 1) / 2) {
    case 3: launch(gemm_ring_kernel<2, 4, 3, 1, 8, 2>, grid, 512, 0, s, A, W, C, M, N, K, ldc, kps, rm); break;
    case 4: launch(gemm_ring_kernel<2, 4, 4, 1, 8, 2>, grid, 512, 0, s, A, W, C, M, N, K, ldc, kps, rm); break;
  }
}

template <int NT, int R, int AD>
static void launch_ring(int mt, dim3 grid, const uint16_t *A, const uint16_t *W, float *C, int M,
                        int N, int K, int ldc, int kps, RowMaxOut rm, hipStream_t s) {
  switch (mt) {
#define WISP_RING_CASE(X) \
  case X: launch(gemm_ring_kernel<1, 4, X, NT, R, AD>, grid, 256, 0, s, A, W, C, M, N, K, ldc, kps, rm); break;
    WISP_RING_CASE(1)
    WISP_RING_CASE(2)
    WISP_RING_CASE(3)
    WISP_RING_CASE(4)
    WISP_RING_CASE(5)
    WISP_RING_CASE(6)
    WISP_RING_CASE(7)
    WISP_RING_CASE(8)
#undef WISP_RING_CASE
  }
}

void gemm_bf16(const uint16_t *A, const uint16_t *W, float *C, int M, int N, int K, int ldc,
               const GemmCfg &cfg, hipStream_t s, RowMaxOut rm, SwigluOut sw) {
  if (cfg.kind == 4) {
    gemm_bf16_tile(A, W, C, M, N, K, ldc, cfg.variant, cfg.kf_per_split / tile_shape(cfg.variant).ks, rm, s, sw);
    return;
  }
  dim3 grid(((N + cfg.bn - 1) / cfg.bn) * cfg.splits, cfg.rb, 1);
  if (cfg.kind == 1)
    launch_ring<1, 8, kNarrowAD>(cfg.mt, grid, A, W, C, M, N, K, ldc, cfg.kf_per_split, rm, s);
  else if (cfg.kind == 3)
    launch_ring_paired(cfg.mt, grid, A, W, C, M, N, K, ldc, cfg.kf_per_split, rm, s);
  else
    launch_ring<2, 4, 2>(cfg.mt, grid, A, W, C, M, N, K, ldc, cfg.kf_per_split, rm, s);
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
  launch(gemm_f32_kernel, grid, 256, 0, s, A, W, C, M, N, K, ldc);
}

// ---------------------------------------------------------------------------------------
// weight packing: natural [rows][cols] -> 32x16 fragments
// ---------------------------------------------------------------------------------------
__global__ void pack_bf16_kernel(uint16_t *__restrict__ dst, const uint16_t *__restrict__ src,
                                 int rows, int cols, int blk_mul, int blk_add) {
  // one thread per (row, 8-column chunk): 16 contiguous bytes in, 16 contiguous bytes out;
  // source row r goes to packed row ((r / 32) * blk_mul + blk_add) * 32 + r % 32
  const int64_t chunks = (int64_t)rows * (cols / 8);
  for (int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; c < chunks;
       c += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = c / (cols / 8), k = (c % (cols / 8)) * 8;
    const int64_t rd = ((r >> 5) * blk_mul + blk_add) * 32 + (r & 31);
    const uint4 v = *reinterpret_cast<const uint4 *>(src + r * cols + k);
    *reinterpret_cast<uint4 *>(dst + packed_off(rd, k, cols)) = v;
  }
}

static void pack_rows(uint16_t *dst, const uint16_t *src, int rows, int cols, int blk_mul, int blk_add,
                      hipStream_t s) {
  const int64_t chunks = (int64_t)rows * (cols / 8);
  int blocks = (int)((chunks + 255) / 256);
  if (blocks > 65535) blocks = 65535;
  launch(pack_bf16_kernel, blocks, 256, 0, s, dst, src, rows, cols, blk_mul, blk_add);
}

void pack_linear_bf16(uint16_t *dst, const uint16_t *src, int rows, int cols, hipStream_t s) {
  pack_rows(dst, src, rows, cols, 1, 0, s);
}

void pack_gate_up_bf16(uint16_t *dst, const uint16_t *gate, const uint16_t *up, int F, int d, hipStream_t s) {
  pack_rows(dst, gate, F, d, 2, 0, s);
  pack_rows(dst, up, F, d, 2, 1, s);
}

}  // namespace wisp
