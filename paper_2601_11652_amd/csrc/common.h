// Device-side helpers shared by the gfx950 kernels of the verification step.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wisp {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kPage = 16;
constexpr int kWave = 64;

// ---------------------------------------------------------------------------------------
// bf16 storage (uint16 bit patterns), round to nearest even; inputs are finite
// ---------------------------------------------------------------------------------------
__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ uint32_t pack2bf(float a, float b) {
  return (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
}

// the same rounding (nearest even) by gfx950's v_cvt_pk_bf16_f32, for finite values
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack2bf_rne(float a, float b) {
  const bf16x2_t v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

template <typename T> struct Act;
template <> struct Act<float> {
  static __device__ __forceinline__ float load(const float *p, int64_t i) { return p[i]; }
  static __device__ __forceinline__ void store(float *p, int64_t i, float v) { p[i] = v; }
};
template <> struct Act<uint16_t> {
  static __device__ __forceinline__ float load(const uint16_t *p, int64_t i) { return bf2f(p[i]); }
  static __device__ __forceinline__ void store(uint16_t *p, int64_t i, float v) { p[i] = f2bf(v); }
};

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// 16-byte loads.  `ld16` is a plain cached load; `ld16_stream` marks data read once
// (the weight stream) as non-temporal so it does not evict reused data from the caches.
__device__ __forceinline__ uint4 ld16(const void *p) {
  const u32x4 v = *reinterpret_cast<const u32x4 *>(p);
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint4 ld16_stream(const void *p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
// zero unless `ok` (the load itself is issued unconditionally from a valid address)
__device__ __forceinline__ uint4 keep_if(bool ok, uint4 v) {
  return ok ? v : make_uint4(0, 0, 0, 0);
}

// ---------------------------------------------------------------------------------------
// Cross-row reductions of a wave (rows = 16-lane groups) on the VALU: gfx950's
// v_permlane16_swap / v_permlane32_swap exchange rows between two registers, so combining
// both outputs reduces over lanes l and l ^ 16 (or l ^ 32) without a trip through LDS.
// Each lane ends with the same value as a shuffle-based reduction (the pairwise
// combination is commutative).
// ---------------------------------------------------------------------------------------
__device__ __forceinline__ float xor16_max(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor32_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor16_sum(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float xor32_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// ---------------------------------------------------------------------------------------
// KV page layouts (one page = 16 slots x hd of one block and kv head)
// ---------------------------------------------------------------------------------------
// K: slots split by bit 2 into two groups of 8, each group's 32-dim chunk contiguous;
// V: each dim's 8 consecutive slots contiguous (one 16-byte operand per lane)
__device__ __forceinline__ int k_page_off(int slot, int e) {
  return (((e >> 5) * 2 + ((slot >> 2) & 1)) * 4 + ((e & 31) >> 3)) * 64 + ((slot >> 3) * 4 + (slot & 3)) * 8 +
         (e & 7);
}
__device__ __forceinline__ int v_page_off(int slot, int e) {
  return ((e >> 4) * 2 + (slot >> 3)) * 128 + (e & 15) * 8 + (slot & 7);
}

// Packed GEMM-operand layout: 32 x 16 fragments, fragment (rb, kb) of a matrix with K
// columns at ((rb * K/16 + kb) * 512); lane l holds row rb*32 + l%32, columns
// kb*16 + (l/32)*8 + 0..7.
__device__ __forceinline__ int64_t packed_off(int64_t r, int64_t c, int64_t K) {
  int64_t rb = r >> 5, kb = c >> 4;
  int64_t lane = (r & 31) + 32 * ((c & 15) >> 3);
  return ((rb * (K >> 4) + kb) * 64 + lane) * 8 + (c & 7);
}

// ---------------------------------------------------------------------------------------
// Philox4x32-10 (Salmon et al., SC'11) and the uniform draw of the verification stream
// ---------------------------------------------------------------------------------------
struct Philox4 {
  uint32_t v[4];
};

__device__ __forceinline__ Philox4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                                uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    uint32_t lo0 = 0xD2511F53u * c0, hi0 = __umulhi(0xD2511F53u, c0);
    uint32_t lo1 = 0xCD9E8D57u * c2, hi1 = __umulhi(0xCD9E8D57u, c2);
    uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  Philox4 o;
  o.v[0] = c0;
  o.v[1] = c1;
  o.v[2] = c2;
  o.v[3] = c3;
  return o;
}

// (2 * (w >> 9) + 1) * 2^-24: exact in fp32, strictly inside (0, 1)
__device__ __forceinline__ float uniform_from_word(uint32_t w) {
  return (float)(((w >> 9) << 1) | 1u) * 5.9604644775390625e-8f;
}

constexpr uint32_t kTagAccept = 1u;
constexpr uint32_t kTagRace = 2u;

// ---------------------------------------------------------------------------------------
// Optional output of a single-K-range projection (the LM head): per row and output tile of
// the GEMM's tile width in columns, the row's maximum over the tile and the first column
// holding it, m[row * tiles + tile]; m == NULL: not computed.
// ---------------------------------------------------------------------------------------
struct RowMaxOut {
  float *m;
  int32_t *i;
  int tiles;
};

// The gate/up projection's epilogue output: silu(gate) * up of each row, stored as bf16
// in the fragment-packed input layout of the down projection (K = F).
struct SwigluOut {
  uint16_t *out;
  int F;
};
// SwiGLU's elementwise step, shared by the SwiGLU kernel and the GEMM epilogue so that both
// give bit-identical results
__device__ __forceinline__ float silu_mul(float g, float u) { return g / (1.0f + expf(-g)) * u; }

// Each row's maximum over one output tile's columns, and the first column holding it, from
// the fp32 accumulators just stored (the LM head's logits).  Lane l of a wave holds column
// l % 32 of each of its fragments for rows 4 (l / 32) + 8 (e / 4) + e % 4; a row's values
// are reduced over the wave's fragments, then over the 32 lanes of its half-wave
// (butterfly), then over the WGN waves of the tile's column range through LDS, in column
// order.  Ties keep the smaller column.  `sh` holds WGN x (WGM * MTW * 32) values and as
// many columns.
template <int WGM, int WGN, int MTW, int NTW>
__device__ __forceinline__ void tile_row_max(const floatx16 (&acc)[MTW][NTW], float *sh, int nb_first, int NF, int N,
                                             int M, int row0, int wrf, int wn, int tile, RowMaxOut rm) {
  constexpr int ROWS = WGM * MTW * 32;
  const int lane = threadIdx.x & 63;
  int *shc = reinterpret_cast<int *>(sh + WGN * ROWS);
#pragma unroll
  for (int i = 0; i < MTW; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      float bv = -INFINITY;
      int bc = 0x7FFFFFFF;
#pragma unroll
      for (int j = 0; j < NTW; ++j) {
        const int col = (nb_first + j) * 32 + (lane & 31);
        if (nb_first + j < NF && col < N && acc[i][j][e] > bv) {
          bv = acc[i][j][e];
          bc = col;
        }
      }
#pragma unroll
      for (int o = 1; o < 32; o <<= 1) {
        const float ov = __shfl_xor(bv, o);
        const int oc = __shfl_xor(bc, o);
        if (ov > bv || (ov == bv && oc < bc)) {
          bv = ov;
          bc = oc;
        }
      }
      if ((lane & 31) == 0) {
        const int lr = (wrf + i) * 32 + 4 * (lane >> 5) + 8 * (e >> 2) + (e & 3);
        sh[wn * ROWS + lr] = bv;
        shc[wn * ROWS + lr] = bc;
      }
    }
  __syncthreads();
  for (int lr = threadIdx.x; lr < ROWS; lr += blockDim.x) {
    const int row = row0 + lr;
    if (row >= M) continue;
    float bv = sh[lr];
    int bc = shc[lr];
    for (int w = 1; w < WGN; ++w) {
      const float ov = sh[w * ROWS + lr];
      const int oc = shc[w * ROWS + lr];
      if (ov > bv || (ov == bv && oc < bc)) {
        bv = ov;
        bc = oc;
      }
    }
    rm.m[(int64_t)row * rm.tiles + tile] = bv;
    rm.i[(int64_t)row * rm.tiles + tile] = bc;
  }
}

// ---------------------------------------------------------------------------------------
// error word bits (kept in the first bytes of the workspace)
// ---------------------------------------------------------------------------------------
constexpr int kErrToken = 1;
constexpr int kErrBlock = 2;

__device__ __forceinline__ void flag_error(int *err, int bit) { atomicOr(err, bit); }

}  // namespace wisp
