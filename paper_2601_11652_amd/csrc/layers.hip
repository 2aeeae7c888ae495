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
  rope_table_kernel<<<(n + 255) / 256, 256, 0, s>>>(d.row_pos, cs, M, hd, base);
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
  embed_norm_kernel<T><<<M, 256, dm * sizeof(float), s>>>(d, embed, gain, tokens, h, xn, packed, dm, V, eps);
}

template <typename T>
__global__ __launch_bounds__(256) void resid_norm_kernel(const float *__restrict__ part, int splits,
                                                         float *__restrict__ h,
                                                         const T *__restrict__ gain,
                                                         T *__restrict__ xn, bool packed, int M,
                                                         int dm, float eps) {
  __shared__ float sh[4];
  extern __shared__ float row[];
  const int r = blockIdx.x;
  float *hr = h + (int64_t)r * dm;
  for (int c = threadIdx.x * 4; c < dm; c += 256 * 4) {
    const float4 acc = sum_splits4(part + (int64_t)r * dm + c, (int64_t)M * dm, splits);
    float4 v = *reinterpret_cast<const float4 *>(hr + c);
    v.x += acc.x;
    v.y += acc.y;
    v.z += acc.z;
    v.w += acc.w;
    *reinterpret_cast<float4 *>(hr + c) = v;
    *reinterpret_cast<float4 *>(row + c) = v;
  }
  __syncthreads();
  norm_store_row<T>(row, gain, xn, packed, r, dm, eps, sh);
}

template <typename T>
void resid_norm(const float *part, int splits, float *h, const T *gain, T *xn, bool packed, int M,
                int dm, float eps, hipStream_t s) {
  resid_norm_kernel<T><<<M, 256, dm * sizeof(float), s>>>(part, splits, h, gain, xn, packed, M, dm, eps);
}

// ---------------------------------------------------------------------------------------
// qkv partials -> RoPE (rotate-half) -> q buffer, k/v appended into the pages in place
// ---------------------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void qkv_rope_append_kernel(StepDesc d, const float *__restrict__ part,
                                                              int splits, const float *__restrict__ cs,
                                                              T *__restrict__ q, T *__restrict__ k_pool,
                                                              T *__restrict__ v_pool, int M, int nq,
                                                              int nkv, int hd) {
  extern __shared__ float row[];   // the row's summed q|k|v projections
  const int r = blockIdx.x;
  const int N = (nq + 2 * nkv) * hd;
  const int h2 = hd / 2;
  for (int c = threadIdx.x * 4; c < N; c += 256 * 4)
    *reinterpret_cast<float4 *>(row + c) = sum_splits4(part + (int64_t)r * N + c, (int64_t)M * N, splits);
  __syncthreads();
  const int req = d.row_req[r], pos = d.row_pos[r];
  const int blk = d.page_table[(int64_t)req * d.pt_stride + pos / kPage];
  const bool blk_ok = blk >= 0 && blk < d.n_blocks;
  if (!blk_ok && threadIdx.x == 0) flag_error(d.err, kErrBlock);
  const int slot = pos % kPage;
  const int page_elems = kPage * hd;
  const float *csr = cs + (int64_t)r * hd;   // [h2][2]
  // rotated pairs (i, i + hd/2): q heads then k heads
  for (int p = threadIdx.x; p < (nq + nkv) * h2; p += 256) {
    const int head = p / h2, i = p % h2;
    const float x1 = row[head * hd + i], x2 = row[head * hd + i + h2];
    const float c = csr[2 * i], sn = csr[2 * i + 1];
    const float y1 = x1 * c - x2 * sn;
    const float y2 = x2 * c + x1 * sn;
    if (head < nq) {
      Act<T>::store(q, ((int64_t)r * nq + head) * hd + i, y1);
      Act<T>::store(q, ((int64_t)r * nq + head) * hd + i + h2, y2);
    } else if (blk_ok) {
      const int kh = head - nq;
      T *pg = k_pool + ((int64_t)blk * nkv + kh) * page_elems;
      Act<T>::store(pg, k_page_off(slot, i), y1);
      Act<T>::store(pg, k_page_off(slot, i + h2), y2);
    }
  }
  if (blk_ok) {
    for (int e = threadIdx.x; e < nkv * hd; e += 256) {
      const int kh = e / hd, dim = e % hd;
      T *pg = v_pool + ((int64_t)blk * nkv + kh) * page_elems;
      Act<T>::store(pg, v_page_off(slot, dim), row[(nq + nkv) * hd + e]);
    }
  }
}

template <typename T>
void qkv_rope_append(const StepDesc &d, const float *part, int splits, const float *cs, T *q,
                     T *k_pool, T *v_pool, int M, int nq, int nkv, int hd, hipStream_t s) {
  const int N = (nq + 2 * nkv) * hd;
  qkv_rope_append_kernel<T><<<M, 256, N * sizeof(float), s>>>(d, part, splits, cs, q, k_pool, v_pool, M, nq, nkv, hd);
}

// ---------------------------------------------------------------------------------------
// SwiGLU: silu(gate) * up, gate/up are columns [0, F) and [F, 2F) of the partials
// ---------------------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void swiglu_kernel(const float *__restrict__ part, int splits,
                                                     T *__restrict__ out, bool packed, int M, int F) {
  const int64_t chunks = (int64_t)M * (F / 8);
  const int64_t stride = (int64_t)M * 2 * F;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < chunks;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = t / (F / 8), c = (t % (F / 8)) * 8;
    const float *pr = part + r * 2 * F;
    float4 g[2], u[2];
    g[0] = sum_splits4(pr + c, stride, splits);
    g[1] = sum_splits4(pr + c + 4, stride, splits);
    u[0] = sum_splits4(pr + F + c, stride, splits);
    u[1] = sum_splits4(pr + F + c + 4, stride, splits);
    const float gv[8] = {g[0].x, g[0].y, g[0].z, g[0].w, g[1].x, g[1].y, g[1].z, g[1].w};
    const float uv[8] = {u[0].x, u[0].y, u[0].z, u[0].w, u[1].x, u[1].y, u[1].z, u[1].w};
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = gv[e] / (1.0f + expf(-gv[e])) * uv[e];
    store8<T>(out, packed, r, c, F, v);
  }
}

template <typename T>
void swiglu(const float *part, int splits, T *out, bool packed, int M, int F, hipStream_t s) {
  const int64_t chunks = (int64_t)M * (F / 8);
  int blocks = (int)((chunks + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  swiglu_kernel<T><<<blocks, 256, 0, s>>>(part, splits, out, packed, M, F);
}

template void embed_norm<float>(const StepDesc &, const float *, const float *, const int32_t *,
                                float *, float *, bool, int, int, int, float, hipStream_t);
template void embed_norm<uint16_t>(const StepDesc &, const uint16_t *, const uint16_t *,
                                   const int32_t *, float *, uint16_t *, bool, int, int, int, float,
                                   hipStream_t);
template void resid_norm<float>(const float *, int, float *, const float *, float *, bool, int, int,
                                float, hipStream_t);
template void resid_norm<uint16_t>(const float *, int, float *, const uint16_t *, uint16_t *, bool,
                                   int, int, float, hipStream_t);
template void qkv_rope_append<float>(const StepDesc &, const float *, int, const float *, float *,
                                     float *, float *, int, int, int, int, hipStream_t);
template void qkv_rope_append<uint16_t>(const StepDesc &, const float *, int, const float *,
                                        uint16_t *, uint16_t *, uint16_t *, int, int, int, int,
                                        hipStream_t);
template void swiglu<float>(const float *, int, float *, bool, int, int, hipStream_t);
template void swiglu<uint16_t>(const float *, int, uint16_t *, bool, int, int, hipStream_t);

}  // namespace wisp
