// Per-row kernels of the verification step: embedding + RMSNorm, the fixed-order sum of
// split-K partials fused with residual add + RMSNorm, RoPE + in-place KV append
// (Sec. 4.5: the new rows' K/V are written into their pages at ctx_len .. ctx_len+gamma),
// and SwiGLU.  Activations that feed a bf16 GEMM are written straight into the packed
// 32x16-fragment layout the GEMM streams; fp32 models keep row-major activations.
#include "common.h"
#include "kernels.h"

namespace wisp {

__device__ __forceinline__ float block_sum_256(float v, float *sh) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  return sh[0] + sh[1] + sh[2] + sh[3];
}

// store 8 consecutive activation columns c..c+7 of row r
template <typename T>
__device__ __forceinline__ void store8(T *out, bool packed, int64_t r, int64_t c, int64_t K,
                                      const float *v);
template <>
__device__ __forceinline__ void store8<float>(float *out, bool, int64_t r, int64_t c, int64_t K,
                                             const float *v) {
#pragma unroll
  for (int e = 0; e < 8; ++e) out[r * K + c + e] = v[e];
}
template <>
__device__ __forceinline__ void store8<uint16_t>(uint16_t *out, bool packed, int64_t r, int64_t c,
                                                int64_t K, const float *v) {
  uint4 w;
  w.x = pack2bf(v[0], v[1]);
  w.y = pack2bf(v[2], v[3]);
  w.z = pack2bf(v[4], v[5]);
  w.w = pack2bf(v[6], v[7]);
  const int64_t o = packed ? packed_off(r, c, K) : r * K + c;
  *reinterpret_cast<uint4 *>(out + o) = w;
}

// Sum of the K-split partials of 4 consecutive fp32 columns, in fixed split order.  All
// split loads are issued before the first add so their latencies overlap.
constexpr int kMaxSplits = 16;
__device__ __forceinline__ float4 sum_splits4(const float *__restrict__ p, int64_t stride, int splits) {
  float4 v[kMaxSplits];
#pragma unroll
  for (int z = 0; z < kMaxSplits; ++z)
    if (z < splits) v[z] = *reinterpret_cast<const float4 *>(p + z * stride);
  float4 a = v[0];
#pragma unroll
  for (int z = 1; z < kMaxSplits; ++z)
    if (z < splits) {
      a.x += v[z].x;
      a.y += v[z].y;
      a.z += v[z].z;
      a.w += v[z].w;
    }
  return a;
}

// ---------------------------------------------------------------------------------------
__global__ void rope_table_kernel(const int32_t *__restrict__ row_pos, float *__restrict__ cs, int M,
                                  int hd, float base) {
  const int h2 = hd / 2;
  const int n = M * h2;
  for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < n; t += gridDim.x * blockDim.x) {
    const int r = t / h2, i = t % h2;
    const double inv = pow((double)base, -2.0 * i / hd);
    const double ang = (double)row_pos[r] * inv;
    cs[2 * t] = (float)cos(ang);
    cs[2 * t + 1] = (float)sin(ang);
  }
}

void rope_table(const StepDesc &d, float *cs, int M, int hd, float base, hipStream_t s) {
  const int n = M * hd / 2;
  launch(rope_table_kernel, (n + 255) / 256, 256, 0, s, d.row_pos, cs, M, hd, base);
}

// ---------------------------------------------------------------------------------------
// RMSNorm of the fp32 row staged in LDS (`hrow`), y = x / rms * g
// ---------------------------------------------------------------------------------------
template <typename T>
__device__ void norm_store_row(const float *__restrict__ hrow, const T *__restrict__ gain,
                               T *__restrict__ xn, bool packed, int64_t r, int dm, float eps,
                               float *sh) {
  float ss = 0.f;
  for (int c = threadIdx.x; c < dm; c += 256) ss += hrow[c] * hrow[c];
  ss = block_sum_256(ss, sh);
  const float inv = 1.0f / sqrtf(ss / (float)dm + eps);
  for (int c8 = threadIdx.x * 8; c8 < dm; c8 += 256 * 8) {
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = hrow[c8 + e] * inv * Act<T>::load(gain, c8 + e);
    store8<T>(xn, packed, r, c8, dm, v);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void embed_norm_kernel(StepDesc d, const T *__restrict__ embed,
                                                         const T *__restrict__ gain,
                                                         const int32_t *__restrict__ tokens,
                                                         float *__restrict__ h, T *__restrict__ xn,
                                                         bool packed, int dm, int V, float eps) {
  __shared__ float sh[4];
  extern __shared__ float row[];
  const int r = blockIdx.x;
  int tok = tokens[r];
  if (tok < 0 || tok >= V) {
    if (threadIdx.x == 0) flag_error(d.err, kErrToken);
    tok = 0;
  }
  float *hr = h + (int64_t)r * dm;
  for (int c = threadIdx.x; c < dm; c += 256) {
    const float v = Act<T>::load(embed, (int64_t)tok * dm + c);
    hr[c] = v;
    row[c] = v;
  }
  __syncthreads();
  norm_store_row<T>(row, gain, xn, packed, r, dm, eps, sh);
}

template <typename T>
void embed_norm(const StepDesc &d, const T *embed, const T *gain, const int32_t *tokens, float *h,
                T *xn, bool packed, int M, int dm, int V, float eps, hipStream_t s) {
  launch(embed_norm_kernel<T>, M, 256, dm * sizeof(float), s, d, embed, gain, tokens, h, xn, packed, dm, V, eps);
}

// Fixed-order sum over the threads of a block of up to 1024 (waves reduce by shuffles,
// then wave sums are added in wave order).
__device__ __forceinline__ float block_sum(float v, float *sh) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6, nw = (blockDim.x + 63) >> 6;
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += sh[i];
  return t;
}

// One row per workgroup, 8 columns per thread: every split partial and the residual are
// loaded in one round, the new residual stays in registers for the norm.
template <typename T>
__global__ __launch_bounds__(1024) void resid_norm_kernel(const float *__restrict__ part, int splits,
                                                          float *__restrict__ h,
                                                          const T *__restrict__ gain,
                                                          T *__restrict__ xn, bool packed, int M,
                                                          int dm, float eps,
                                                          const int32_t *__restrict__ rows) {
  __shared__ float sh[16];
  const int ro = blockIdx.x;                 // output row
  const int r = rows ? rows[ro] : ro;        // source row
  const int c = threadIdx.x * 8;
  const bool on = c < dm;
  float v[8];
  float ss = 0.f;
  if (on) {
    const float *p = part + (int64_t)r * dm + c;
    const int64_t stride = (int64_t)M * dm;
    const float4 a0 = sum_splits4(p, stride, splits);
    const float4 a1 = sum_splits4(p + 4, stride, splits);
    float *hr = h + (int64_t)r * dm + c;
    const float4 h0 = *reinterpret_cast<const float4 *>(hr);
    const float4 h1 = *reinterpret_cast<const float4 *>(hr + 4);
    v[0] = h0.x + a0.x; v[1] = h0.y + a0.y; v[2] = h0.z + a0.z; v[3] = h0.w + a0.w;
    v[4] = h1.x + a1.x; v[5] = h1.y + a1.y; v[6] = h1.z + a1.z; v[7] = h1.w + a1.w;
    *reinterpret_cast<float4 *>(hr) = make_float4(v[0], v[1], v[2], v[3]);
    *reinterpret_cast<float4 *>(hr + 4) = make_float4(v[4], v[5], v[6], v[7]);
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += v[e] * v[e];
  }
  ss = block_sum(ss, sh);
  if (!on) return;
  const float inv = 1.0f / sqrtf(ss / (float)dm + eps);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = v[e] * inv * Act<T>::load(gain, c + e);
  store8<T>(xn, packed, ro, c, dm, v);
}

template <typename T>
void resid_norm(const float *part, int splits, float *h, const T *gain, T *xn, bool packed, int M,
                int dm, float eps, hipStream_t s, const int32_t *rows, int n_out) {
  const int threads = ((dm / 8 + 63) / 64) * 64;   // dm <= 8192
  const int n = rows ? n_out : M;
  if (n <= 0) return;
  launch(resid_norm_kernel<T>, n, threads, 0, s, part, splits, h, gain, xn, packed, M, dm, eps, rows);
}

__global__ void gather_ints_kernel(const int32_t *__restrict__ src, const int32_t *__restrict__ idx, int n,
                                   int32_t *__restrict__ dst) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src[idx[i]];
}

void gather_ints(const int32_t *src, const int32_t *idx, int n, int32_t *dst, hipStream_t s) {
  if (n > 0) launch(gather_ints_kernel, (n + 255) / 256, 256, 0, s, src, idx, n, dst);
}

// ---------------------------------------------------------------------------------------
// qkv partials -> RoPE (rotate-half) -> q buffer, k/v appended into the pages in place
// ---------------------------------------------------------------------------------------
// Grid (row, group of 8 heads); each thread owns 8 consecutive dims of one head.  The
// rotate-half partner (dims i and i + hd/2) belongs to the thread hd/16 places further
// round the same head; partners are exchanged through LDS, which pairs the right threads
// for every head_dim (a head need not sit inside one wave, nor at a power-of-two lane
// offset).  q and K are written as 16-byte stores (8 consecutive dims are contiguous in
// the K page layout), V element by element.
constexpr int kRopeHeadsPerBlock = 8;

template <typename T>
__device__ __forceinline__ void store8_contig(T *p, const float *v);
template <>
__device__ __forceinline__ void store8_contig<float>(float *p, const float *v) {
  *reinterpret_cast<float4 *>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4 *>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
template <>
__device__ __forceinline__ void store8_contig<uint16_t>(uint16_t *p, const float *v) {
  *reinterpret_cast<uint4 *>(p) = make_uint4(pack2bf(v[0], v[1]), pack2bf(v[2], v[3]),
                                             pack2bf(v[4], v[5]), pack2bf(v[6], v[7]));
}

template <typename T>
__global__ __launch_bounds__(256) void qkv_rope_append_kernel(StepDesc d, const float *__restrict__ part,
                                                              int splits, const float *__restrict__ cs,
                                                              T *__restrict__ q, T *__restrict__ k_pool,
                                                              T *__restrict__ v_pool, int M, int nq,
                                                              int nkv, int hd) {
  const int r = blockIdx.x;
  const int tph = hd / 8;                          // threads per head
  const int head = blockIdx.y * kRopeHeadsPerBlock + threadIdx.x / tph;
  const int nh = nq + 2 * nkv;
  const int i0 = (threadIdx.x % tph) * 8;          // first dim of this thread
  const int h2 = hd / 2;
  const int N = nh * hd;
  __shared__ float xch[kRopeHeadsPerBlock * 256];   // 8 values per thread, hd <= 256
  float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (head < nh) {
    const float *p = part + (int64_t)r * N + head * hd + i0;
    const int64_t stride = (int64_t)M * N;
    const float4 a0 = sum_splits4(p, stride, splits);
    const float4 a1 = sum_splits4(p + 4, stride, splits);
    v[0] = a0.x; v[1] = a0.y; v[2] = a0.z; v[3] = a0.w;
    v[4] = a1.x; v[5] = a1.y; v[6] = a1.z; v[7] = a1.w;
  }
  // rotate-half partner values: thread t of a head pairs with thread (t + tph/2) mod tph
#pragma unroll
  for (int e = 0; e < 8; ++e) xch[threadIdx.x * 8 + e] = v[e];
  __syncthreads();
  const int partner = (threadIdx.x / tph) * tph + (threadIdx.x % tph + tph / 2) % tph;
  float w[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) w[e] = xch[partner * 8 + e];
  if (head >= nh) return;
  const int req = d.row_req[r], pos = d.row_pos[r];
  if (head < nq + nkv) {   // RoPE on q and k heads
    const float *csr = cs + (int64_t)r * hd;   // [h2][2]
    const bool lo = i0 < h2;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int i = (lo ? i0 : i0 - h2) + e;
      const float c = csr[2 * i], sn = csr[2 * i + 1];
      v[e] = lo ? v[e] * c - w[e] * sn : v[e] * c + w[e] * sn;
    }
  }
  if (head < nq) {
    store8_contig<T>(q + ((int64_t)r * nq + head) * hd + i0, v);
    return;
  }
  const int blk = d.page_table[(int64_t)req * d.pt_stride + pos / kPage];
  if (blk < 0 || blk >= d.n_blocks) {
    if (threadIdx.x % tph == 0) flag_error(d.err, kErrBlock);
    return;
  }
  const int slot = pos % kPage;
  const int page_elems = kPage * hd;
  if (head < nq + nkv) {
    T *pg = k_pool + ((int64_t)blk * nkv + (head - nq)) * page_elems;
    store8_contig<T>(pg + k_page_off(slot, i0), v);
  } else {
    T *pg = v_pool + ((int64_t)blk * nkv + (head - nq - nkv)) * page_elems;
#pragma unroll
    for (int e = 0; e < 8; ++e) Act<T>::store(pg, v_page_off(slot, i0 + e), v[e]);
  }
}

template <typename T>
void qkv_rope_append(const StepDesc &d, const float *part, int splits, const float *cs, T *q,
                     T *k_pool, T *v_pool, int M, int nq, int nkv, int hd, hipStream_t s) {
  const int nh = nq + 2 * nkv;
  dim3 grid(M, (nh + kRopeHeadsPerBlock - 1) / kRopeHeadsPerBlock);
  launch(qkv_rope_append_kernel<T>, grid, kRopeHeadsPerBlock * hd / 8, 0, s, d, part, splits, cs, q, k_pool, v_pool, M,
                                                                        nq, nkv, hd);
}

// ---------------------------------------------------------------------------------------
// SwiGLU: silu(gate) * up.  Gate/up partials are either stacked (columns [0, F) and
// [F, 2F): the fp32 path) or interleaved by 32-column fragments (bf16 weights packed by
// wisp_pack_gate_up: fragment 2b holds gate columns 32b .. 32b + 31, fragment 2b + 1 the
// up columns of the same b)
// ---------------------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void swiglu_kernel(const float *__restrict__ part, int splits,
                                                     T *__restrict__ out, bool packed, int M, int F,
                                                     bool interleaved) {
  const int64_t chunks = (int64_t)M * (F / 8);
  const int64_t stride = (int64_t)M * 2 * F;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < chunks;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = t / (F / 8), c = (t % (F / 8)) * 8;
    const float *pr = part + r * 2 * F;
    const int64_t gc = interleaved ? (c / 32) * 64 + c % 32 : c;
    const int64_t uc = interleaved ? gc + 32 : F + c;
    float4 g[2], u[2];
    g[0] = sum_splits4(pr + gc, stride, splits);
    g[1] = sum_splits4(pr + gc + 4, stride, splits);
    u[0] = sum_splits4(pr + uc, stride, splits);
    u[1] = sum_splits4(pr + uc + 4, stride, splits);
    const float gv[8] = {g[0].x, g[0].y, g[0].z, g[0].w, g[1].x, g[1].y, g[1].z, g[1].w};
    const float uv[8] = {u[0].x, u[0].y, u[0].z, u[0].w, u[1].x, u[1].y, u[1].z, u[1].w};
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = silu_mul(gv[e], uv[e]);
    store8<T>(out, packed, r, c, F, v);
  }
}

template <typename T>
void swiglu(const float *part, int splits, T *out, bool packed, int M, int F, bool interleaved, hipStream_t s) {
  const int64_t chunks = (int64_t)M * (F / 8);
  int blocks = (int)((chunks + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  launch(swiglu_kernel<T>, blocks, 256, 0, s, part, splits, out, packed, M, F, interleaved);
}

template void embed_norm<float>(const StepDesc &, const float *, const float *, const int32_t *,
                                float *, float *, bool, int, int, int, float, hipStream_t);
template void embed_norm<uint16_t>(const StepDesc &, const uint16_t *, const uint16_t *,
                                   const int32_t *, float *, uint16_t *, bool, int, int, int, float,
                                   hipStream_t);
template void resid_norm<float>(const float *, int, float *, const float *, float *, bool, int, int,
                                float, hipStream_t, const int32_t *, int);
template void resid_norm<uint16_t>(const float *, int, float *, const uint16_t *, uint16_t *, bool,
                                   int, int, float, hipStream_t, const int32_t *, int);
template void qkv_rope_append<float>(const StepDesc &, const float *, int, const float *, float *,
                                     float *, float *, int, int, int, int, hipStream_t);
template void qkv_rope_append<uint16_t>(const StepDesc &, const float *, int, const float *,
                                        uint16_t *, uint16_t *, uint16_t *, int, int, int, int,
                                        hipStream_t);
template void swiglu<float>(const float *, int, float *, bool, int, int, bool, hipStream_t);
template void swiglu<uint16_t>(const float *, int, uint16_t *, bool, int, int, bool, hipStream_t);

}  // namespace wisp
