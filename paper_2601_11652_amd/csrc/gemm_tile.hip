// Dense projections of the verification step at large row counts (a prompt's cold start, or
// hundreds of requests in one step): the regime where the GEMMs are bound by the matrix
// cores rather than by the weight stream.
//
// Both operands are fragment-packed (32 x 16 blocks in the lane order of gfx950's
// v_mfma_f32_32x32x16_bf16, 1 KiB contiguous per block), so one global_load_lds_dwordx4
// moves one fragment into LDS in exactly the order the waves read it back (each lane's
// 16 bytes at lane * 16: conflict-free ds_read_b128), without a trip through registers.
// A workgroup of WGM x WGN waves computes a (32 WGM MTW) x (32 WGN NTW) output tile, each
// wave a tile of MTW x NTW fragments; its A and W slices stream through a ring of ST LDS
// stages of KS K-steps, ST - 1 of them in flight while one is consumed.
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace wisp {

// calls f(integral_constant<int, 0>) .. f(integral_constant<int, N - 1>) in order
template <int N, int I = 0, class F>
__device__ __forceinline__ void static_for(F &&f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, I + 1>(f);
  }
}

// One 16-byte-per-lane load from global memory straight into LDS: lane l's 16 bytes land at
// dst + 16 l (dst wave-uniform, passed in M0).  Issued as inline assembly: the compiler then
// inserts no wait of its own before later LDS reads (it would otherwise assume any such
// load in flight may alias them and wait for all of them), and the kernel waits on the
// vector-memory counter itself, counting exactly the loads it issued.  The kernel issues
// no other vector-memory operation while such loads are in flight.
__device__ __forceinline__ void lds_dma16(const void *src, const void *dst) {
  // dst is wave-uniform by construction; readfirstlane makes that visible to the compiler
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void *)dst);
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(src), "s"(m0) : "memory", "m0");
}
// the same for data read once (the weight stream): marked non-temporal, so the caches do
// not keep it at the expense of the activation slices that the other tiles re-read (measured
// on weight-heavy tiles: the weight stream runs about a third faster)
__device__ __forceinline__ void lds_dma16_stream(const void *src, const void *dst) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void *)dst);
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off nt" : : "v"(src), "s"(m0) : "memory", "m0");
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding: vmcnt in bits
// 3:0 and 15:14, expcnt 6:4 and lgkmcnt 11:8 left at their maxima)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

template <int WGM, int WGN, int MTW, int NTW, int KS, int ST, bool RM, bool SW>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_tile_kernel(const uint16_t *__restrict__ A,
                                                        const uint16_t *__restrict__ W,
                                                        float *__restrict__ C, int M, int N, int K,
                                                        int ldc, int tiles_m, int tiles, int per_xcd,
                                                        int kc_split, RowMaxOut rmax, SwigluOut sw) {
  constexpr int NW = WGM * WGN;               // waves
  constexpr int AF = WGM * MTW, BF = WGN * NTW;   // A / W fragments of the tile per K step
  constexpr int SF = (AF + BF) * KS;          // fragments per stage
  static_assert(SF % NW == 0, "every wave issues the same number of loads");
  constexpr int LPW = SF / NW;                // loads per wave per stage
  static_assert((ST - 2) * LPW < 64, "outstanding loads fit the counter");
  // one LDS object per stage: with distinct objects the compiler can tell that a stage's
  // in-flight loads do not alias the stage being read, and inserts no wait for them
  __shared__ __attribute__((aligned(1024))) uint4 lds0[SF][64];
  __shared__ __attribute__((aligned(1024))) uint4 lds1[SF][64];
  __shared__ __attribute__((aligned(1024))) uint4 lds2[SF][64];
  __shared__ __attribute__((aligned(1024))) uint4 lds3[SF][64];
  __shared__ __attribute__((aligned(1024))) uint4 lds4[ST > 4 ? SF : 1][64];
  __shared__ __attribute__((aligned(1024))) uint4 lds5[ST > 5 ? SF : 1][64];
  static_assert(ST >= 2 && ST <= 6, "stage ring of 2 to 6 buffers");
  auto stage = [&](auto b) -> uint4 (*)[64] {
    constexpr int B = decltype(b)::value;
    if constexpr (B == 0) return lds0;
    else if constexpr (B == 1) return lds1;
    else if constexpr (B == 2) return lds2;
    else if constexpr (B == 3) return lds3;
    else if constexpr (B == 4) return lds4;
    else return lds5;
  };

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  const int KF = K >> 4, MF = (M + 31) >> 5, NF = N >> 5;
  const int KC_all = KF / KS;                 // K chunks (K is a multiple of 16 KS)
  // Workgroups are dealt to the 8 XCDs in turn (id mod 8).  Each XCD takes a contiguous run
  // of per_xcd tiles, column-tile major, so the workgroups resident on one XCD share the
  // A row slices and W column slices of few tiles, which its L2 then serves; the mapping
  // only moves traffic between cache levels, results do not depend on it.
  // Work items are (K range, tile) pairs, K range major: an XCD's run mostly shares one K
  // range, i.e. one slice of A, in its L2.  K range z sums chunks [z kc_split, ...) into
  // its own fp32 partial C[z]; the consumer adds the partials in fixed order.
  const int v = (int)(blockIdx.x % 8u) * per_xcd + (int)(blockIdx.x / 8u);
  const int splits = (KC_all + kc_split - 1) / kc_split;
  if (v >= tiles * splits) return;
  const int z = v / tiles, t = v % tiles;
  const int tm = t % tiles_m, tn = t / tiles_m;
  const int kc0 = z * kc_split;
  const int KC = min(KC_all, kc0 + kc_split) - kc0;
  C += (int64_t)z * M * ldc;
  const int rb0 = tm * AF, nb0 = tn * BF;

  // this wave's loads of chunk c into stage buffer b: fragment f of the stage is A block
  // (f / KS, f % KS) for f < AF KS, else W block; fragments past the matrix edge re-read
  // the last block (their products land in rows / columns that are never stored)
  auto issue = [&](int c, auto b) {
    uint4 (*buf)[64] = stage(b);
#pragma unroll
    for (int t = 0; t < LPW; ++t) {
      const int f = wave * LPW + t;
      if (f < AF * KS) {
        const int rb = min(rb0 + f / KS, MF - 1), kb = (kc0 + c) * KS + f % KS;
        lds_dma16(A + ((int64_t)rb * KF + kb) * 512 + lane * 8, &buf[f][0]);
      } else {
        const int g = f - AF * KS;
        const int nb = min(nb0 + g / KS, NF - 1), kb = (kc0 + c) * KS + g % KS;
        lds_dma16_stream(W + ((int64_t)nb * KF + kb) * 512 + lane * 8, &buf[f][0]);
      }
    }
  };

  floatx16 acc[MTW][NTW];
#pragma unroll
  for (int i = 0; i < MTW; ++i)
#pragma unroll
    for (int j = 0; j < NTW; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // this wave's operands of the chunk in stage buffer b, read from LDS into registers
  auto read_ops = [&](auto b, uint4 (&a)[KS][MTW], uint4 (&w)[KS][NTW]) {
    uint4 (*buf)[64] = stage(b);
#pragma unroll
    for (int k = 0; k < KS; ++k) {
#pragma unroll
      for (int i = 0; i < MTW; ++i) a[k][i] = buf[(wm * MTW + i) * KS + k][lane];
#pragma unroll
      for (int j = 0; j < NTW; ++j) w[k][j] = buf[AF * KS + (wn * NTW + j) * KS + k][lane];
    }
  };
  auto products = [&](const uint4 (&a)[KS][MTW], const uint4 (&w)[KS][NTW]) {
#pragma unroll
    for (int k = 0; k < KS; ++k)
#pragma unroll
      for (int i = 0; i < MTW; ++i)
#pragma unroll
        for (int j = 0; j < NTW; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a[k][i]), as_bf16x8(w[k][j]), acc[i][j],
                                                             0, 0, 0);
  };

  static_for<ST - 1>([&](auto sb) {
    if (sb.value < KC) issue(sb.value, sb);
  });
  // one step of the ring: chunk c sits in stage buffer B; the load of chunk c + ST - 1 goes
  // to buffer (B + ST - 1) % ST, freed by chunk c - 1.  With `guarded` false the caller
  // knows c + ST - 1 < KC (steady state), so the step has no conditions: with them the
  // compiler keeps the accumulators of the two paths in different registers and copies
  auto step = [&](int c, auto bc, auto guarded) {
    constexpr int B = decltype(bc)::value;
    constexpr bool G = decltype(guarded)::value;
    // chunk c's loads (this wave's) have landed once at most the later in-flight chunks'
    // remain; at the tail fewer chunks are in flight, so wait for all
    if (!G || c + ST - 2 < KC)
      wait_vmcnt<(ST - 2) * LPW>();
    else
      wait_vmcnt<0>();
    // every wave's loads of chunk c are in LDS, and every wave is done reading chunk c - 1
    // (its reads completed before its last products): a bare barrier, no memory fence
    __builtin_amdgcn_s_barrier();
    if (!G || c + ST - 1 < KC) issue(c + ST - 1, std::integral_constant<int, (B + ST - 1) % ST>{});
    // all of the stage's operands are read up front, so the reads of step k + 1 overlap the
    // products of step k
    uint4 a[KS][MTW], w[KS][NTW];
    read_ops(bc, a, w);
    products(a, w);
  };
  int c = 0;
  for (; c + 2 * ST - 2 < KC; c += ST) static_for<ST>([&](auto bc) { step(c + bc.value, bc, std::false_type{}); });
  for (; c < KC; c += ST)
    static_for<ST>([&](auto bc) {
      if (c + bc.value < KC) step(c + bc.value, bc, std::true_type{});
    });

  wait_vmcnt<0>();
  if constexpr (SW) {
    // gate/up projection with its weights packed by wisp_pack_gate_up: column fragment 2b
    // holds gate columns 32b .. 32b + 31 and fragment 2b + 1 the up columns of the same b,
    // so silu(gate) * up of column j = 32b + (lane % 32) pairs fragments 2b and 2b + 1 at
    // the same lane and accumulator element.  The tile's first fragment is even (BF is).
    static_assert(BF % 2 == 0, "gate/up fragment pairs stay inside one tile");
    auto emit = [&](int i, int nb_gate, const floatx16 &g, const floatx16 &u) {
      if (nb_gate >= NF) return;
      const int rbase = (rb0 + wm * MTW + i) * 32 + 4 * (lane >> 5);
      const int j = (nb_gate >> 1) * 32 + (lane & 31);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = rbase + 8 * (e >> 2) + (e & 3);
        if (row < M) sw.out[packed_off(row, j, sw.F)] = f2bf(silu_mul(g[e], u[e]));
      }
    };
    if constexpr (NTW % 2 == 0) {   // both fragments of a pair in this wave's registers
#pragma unroll
      for (int i = 0; i < MTW; ++i)
#pragma unroll
        for (int q = 0; q < NTW; q += 2) emit(i, nb0 + wn * NTW + q, acc[i][q], acc[i][q + 1]);
    } else {
      // one fragment per wave: wave wn + 1 (odd) holds the up half of wave wn's gate
      // fragment; it hands its accumulators over through LDS, one row fragment at a time
      static_assert(NTW == 1 && WGN % 2 == 0, "gate/up pairs across neighbouring waves");
      static_assert(WGM * (WGN / 2) * 16 * 64 * 4 <= SF * 1024, "the exchange fits one stage buffer");
      float *x = reinterpret_cast<float *>(&lds0[0][0]) + ((wm * (WGN / 2) + (wn >> 1)) * 16) * 64 + lane;
#pragma unroll
      for (int i = 0; i < MTW; ++i) {
        __syncthreads();   // every wave is done with the stage buffers / the previous round
        if (wn & 1) {
#pragma unroll
          for (int e = 0; e < 16; ++e) x[e * 64] = acc[i][0][e];
        }
        __syncthreads();
        if (!(wn & 1)) {
          floatx16 u;
#pragma unroll
          for (int e = 0; e < 16; ++e) u[e] = x[e * 64];
          emit(i, nb0 + wn, acc[i][0], u);
        }
      }
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < MTW; ++i) {
    const int rbase = (rb0 + wm * MTW + i) * 32 + 4 * (lane >> 5);
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
      const int nb = nb0 + wn * NTW + j;
      if (nb >= NF) continue;
      const int col = nb * 32 + (lane & 31);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = rbase + 8 * (e >> 2) + (e & 3);
        if (row < M) C[(int64_t)row * ldc + col] = acc[i][j][e];
      }
    }
  }
  if (RM) {   // LM head: the row maxima of this tile's columns (its own instance: the
             // maxima need registers that the plain projections spend on their tiles)
    __syncthreads();   // every wave is done with the stage buffers (no load is in flight)
    tile_row_max<WGM, WGN, MTW, NTW>(acc, reinterpret_cast<float *>(&lds0[0][0]), nb0 + wn * NTW, NF, N, M,
                                     rb0 * 32, wm * MTW, wn, tn, rmax);
  }
}

template <int WGM, int WGN, int MTW, int NTW, int KS, int ST>
static void launch_tile(const uint16_t *A, const uint16_t *W, float *C, int M, int N, int K, int ldc,
                        RowMaxOut rm, hipStream_t s, int kc_split, SwigluOut sw) {
  static_assert(2 * WGN * WGM * MTW * 32 * 4 <= (WGM * MTW + WGN * NTW) * KS * 1024,
                "the row-maxima exchange fits one stage buffer");
  const int tiles_m = ((M + 31) / 32 + WGM * MTW - 1) / (WGM * MTW);
  const int tiles_n = (N / 32 + WGN * NTW - 1) / (WGN * NTW);
  const int KC = K / (16 * KS);
  const int splits = (KC + kc_split - 1) / kc_split;
  const int tiles = tiles_m * tiles_n, per_xcd = (tiles * splits + 7) / 8;
  if (rm.m)
    launch(gemm_tile_kernel<WGM, WGN, MTW, NTW, KS, ST, true, false>, 8 * per_xcd, 64 * WGM * WGN, 0, s, A, W, C, M,
           N, K, ldc, tiles_m, tiles, per_xcd, kc_split, rm, sw);
  else if (sw.out)
    launch(gemm_tile_kernel<WGM, WGN, MTW, NTW, KS, ST, false, true>, 8 * per_xcd, 64 * WGM * WGN, 0, s, A, W, C, M,
           N, K, ldc, tiles_m, tiles, per_xcd, kc_split, rm, sw);
  else
    launch(gemm_tile_kernel<WGM, WGN, MTW, NTW, KS, ST, false, false>, 8 * per_xcd, 64 * WGM * WGN, 0, s, A, W, C, M,
           N, K, ldc, tiles_m, tiles, per_xcd, kc_split, rm, sw);
}

// Tile shapes (measured at 7-1237 rows of the 8B and 70B projections, cold weights):
// 8 waves in 2 x 4 or 4 x 2 wave tiles of 3 x 1, 3 x 2, 2 x 2 or 4 x 2 fragments, two waves
// per SIMD; the wider the column tile, the fewer times the activation slice is re-read.  At
// 33-128 rows 64 x 128 and 128 x 128 tiles of single-fragment wave tiles; at most 32 rows
// a 32 x 256 tile of 4 waves with a deep K split.  At these row counts the activation slice
// and the fp32 partials are small next to the weights, so the loads are almost all weights.
// The 384 x 128 and 256 x 256 tiles stage one K step per chunk in a ring of 6 (at 300-1237
// rows 0-9% faster than two K steps in a ring of 4, which holds more K in flight: with
// half-size chunks each barrier waits on less).
TileShape tile_shape(int variant) {
  switch (variant) {
    case 1: return {192, 128, 4};
    case 4: return {192, 256, 4};
    case 12: return {384, 128, 1};
    case 13: return {256, 128, 2};
    case 5: return {32, 256, 4};
    case 6: return {64, 128, 4};
    case 7: return {128, 128, 4};
    case 17: return {256, 256, 1};
  }
  return {0, 0, 0};
}

void gemm_bf16_tile(const uint16_t *A, const uint16_t *W, float *C, int M, int N, int K, int ldc, int variant,
                    int kc_split, RowMaxOut rm, hipStream_t s, SwigluOut sw) {
  switch (variant) {
    case 1: launch_tile<2, 4, 3, 1, 4, 3>(A, W, C, M, N, K, ldc, rm, s, kc_split, sw); break;
    case 4: launch_tile<2, 4, 3, 2, 4, 2>(A, W, C, M, N, K, ldc, rm, s, kc_split, sw); break;
    case 12: launch_tile<4, 2, 3, 2, 1, 6>(A, W, C, M, N, K, ldc, rm, s, kc_split, sw); break;
    case 13: launch_tile<4, 2, 2, 2, 2, 4>(A, W, C, M, N, K, ldc, rm, s, kc_split, sw); break;
    case 5: launch_tile<1, 4, 1, 2, 4, 4>(A, W, C, M, N, K, ldc, rm, s, kc_split, sw); break;   // 4 waves
    case 6: launch_tile<2, 4, 1, 1, 4, 4>(A, W, C, M, N, K, ldc, rm, s, kc_split, sw); break;
    case 7: launch_tile<4, 2, 1, 2, 4, 3>(A, W, C, M, N, K, ldc, rm, s, kc_split, sw); break;
    case 17: launch_tile<2, 4, 4, 2, 1, 6>(A, W, C, M, N, K, ldc, rm, s, kc_split, sw); break;
  }
}

}  // namespace wisp
