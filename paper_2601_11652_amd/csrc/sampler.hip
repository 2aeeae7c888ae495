// Acceptance stage of the verification step (Sec. 2.4): Eq. (1) accept draft y_j with
// probability min(1, p/q), Eq. (2) stop at the first rejection R, Eq. (3) emit one extra
// token -- drawn from norm(max(0, p_R - q_R)) after a rejection (the residual that makes
// speculative sampling lossless) and from p after a fully accepted block.
//
// Two kernels per batch: per-row softmax statistics (max and sum of exponentials of
// z = logits / T, a vocabulary-wide two-pass reduction), then one workgroup per request
// runs the sequential accept scan and the vocabulary-wide exponential race that samples
// the extra token (argmax of score - ln(-ln u), no prefix sums, so the result does not
// depend on reduction order).  All random draws come from Philox4x32-10 keyed by the
// seed and counted by (index, row, request, purpose).
#pragma clang fp contract(off)
#include "common.h"
#include "kernels.h"

namespace wisp {

__device__ __forceinline__ Philox4 draw(uint64_t seed, uint32_t c0, uint32_t row, uint32_t req,
                                        uint32_t tag) {
  return philox4x32_10(c0, row, req, tag, (uint32_t)seed, (uint32_t)(seed >> 32));
}

template <typename V, typename F>
__device__ __forceinline__ V block_reduce(V v, V *sh, F op) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = op(v, __shfl_xor(v, o));
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  V r = sh[0];
  for (int w = 1; w < (int)(blockDim.x >> 6); ++w) r = op(r, sh[w]);
  return r;
}

// ---------------------------------------------------------------------------------------
// row statistics: m = max z, S = sum exp(z - m) (fp64 accumulation, rounded to fp32),
// and the first argmax of the logits (greedy decoding)
// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void row_stats_kernel(const float *__restrict__ logits, int V,
                                                        float T, float *__restrict__ row_m,
                                                        float *__restrict__ row_s,
                                                        int32_t *__restrict__ row_amax) {
  __shared__ float shf[4];
  __shared__ double shd[4];
  __shared__ float shv[4];
  __shared__ int shi[4];
  const int64_t r = blockIdx.x;
  const float *l = logits + r * V;
  if (T == 0.f) {
    float bv = -INFINITY;
    int bi = 0x7FFFFFFF;
    for (int k = threadIdx.x; k < V; k += 256) {
      const float v = l[k];
      if (v > bv) {
        bv = v;
        bi = k;
      }
    }
    // (value, index) reduction: larger value wins, smaller index on ties
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(bv, o);
      const int oi = __shfl_xor(bi, o);
      if (ov > bv || (ov == bv && oi < bi)) {
        bv = ov;
        bi = oi;
      }
    }
    if ((threadIdx.x & 63) == 0) {
      shv[threadIdx.x >> 6] = bv;
      shi[threadIdx.x >> 6] = bi;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      bv = shv[0];
      bi = shi[0];
      for (int w = 1; w < 4; ++w)
        if (shv[w] > bv || (shv[w] == bv && shi[w] < bi)) {
          bv = shv[w];
          bi = shi[w];
        }
      row_amax[r] = bi;
      row_m[r] = bv;
      row_s[r] = 1.f;
    }
    return;
  }
  float mx = -INFINITY;
  for (int k = threadIdx.x; k < V; k += 256) mx = fmaxf(mx, l[k] / T);
  mx = block_reduce(mx, shf, [](float a, float b) { return fmaxf(a, b); });
  double sum = 0.0;
  for (int k = threadIdx.x; k < V; k += 256) sum += (double)expf(l[k] / T - mx);
  sum = block_reduce(sum, shd, [](double a, double b) { return a + b; });
  if (threadIdx.x == 0) {
    row_m[r] = mx;
    row_s[r] = (float)sum;
    row_amax[r] = -1;
  }
}

// ---------------------------------------------------------------------------------------
// accept scan + extra-token race, one workgroup per request
// ---------------------------------------------------------------------------------------
__device__ __forceinline__ bool better(float ka, int ia, float kb, int ib) {
  return ka > kb || (ka == kb && ia < ib);
}

__global__ __launch_bounds__(256) void accept_kernel(StepDesc d, int V, const float *__restrict__ logits,
                                                     const int32_t *__restrict__ tokens,
                                                     const float *__restrict__ q, float T,
                                                     uint64_t seed, const float *__restrict__ row_m,
                                                     const float *__restrict__ row_s,
                                                     const int32_t *__restrict__ row_amax,
                                                     int32_t *__restrict__ accept_len,
                                                     int32_t *__restrict__ out_tokens) {
  __shared__ int R_sh;
  __shared__ float shk[2][4];
  __shared__ int shi[2][4];
  __shared__ int shany[4];
  const int i = blockIdx.x;
  const int gam = d.gamma[i], off = d.off[i], doff = d.doff[i];
  const uint32_t req = d.req_id[i];
  if (threadIdx.x == 0) {
    int R = gam + 1;
    for (int j = 1; j <= gam; ++j) {
      int y = tokens[off + j];
      if (y < 0 || y >= V) {
        flag_error(d.err, kErrToken);
        y = 0;
      }
      const int64_t pr = off + j - 1;
      if (T == 0.f) {
        if (y != row_amax[pr]) {
          R = j;
          break;
        }
      } else {
        const float P = expf(logits[pr * V + y] / T - row_m[pr]) / row_s[pr];
        const float Q = q[(int64_t)(doff + j - 1) * V + y];
        const float a = Q > 0.f ? fminf(1.f, P / Q) : (P > 0.f ? 1.f : 0.f);
        const float u = uniform_from_word(draw(seed, 0u, (uint32_t)j, req, kTagAccept).v[0]);
        if (!(u <= a)) {
          R = j;
          break;
        }
      }
    }
    R_sh = R;
  }
  __syncthreads();
  const int R = R_sh, L = R - 1, r = R - 1;
  const int64_t lr = off + r;
  int extra;
  if (T == 0.f) {
    extra = row_amax[lr];
  } else {
    const float *l = logits + lr * V;
    const bool rejected = R <= gam;
    const float *qr = q + (int64_t)(doff + (rejected ? R - 1 : 0)) * V;
    const float m = row_m[lr], S = row_s[lr];
    float kR = -INFINITY, kP = -INFINITY;
    int iR = 0x7FFFFFFF, iP = 0x7FFFFFFF;
    int any = 0;
    for (int k4 = threadIdx.x; k4 * 4 < V; k4 += 256) {
      const Philox4 w = draw(seed, (uint32_t)k4, (uint32_t)r, req, kTagRace);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int k = k4 * 4 + e;
        if (k >= V) break;
        const float z = l[k] / T;
        const float g = logf(-logf(uniform_from_word(w.v[e])));
        const float keyp = z - g;
        if (keyp > kP) {
          kP = keyp;
          iP = k;
        }
        if (rejected) {
          const float p = expf(z - m) / S;
          const float wk = p - qr[k];
          if (wk > 0.f) {
            any = 1;
            const float keyr = logf(wk) - g;
            if (keyr > kR) {
              kR = keyr;
              iR = k;
            }
          }
        }
      }
    }
    // per-thread candidates were visited in ascending k, so strict '>' kept the first
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      float ok = __shfl_xor(kP, o);
      int oi = __shfl_xor(iP, o);
      if (better(ok, oi, kP, iP)) {
        kP = ok;
        iP = oi;
      }
      ok = __shfl_xor(kR, o);
      oi = __shfl_xor(iR, o);
      if (better(ok, oi, kR, iR)) {
        kR = ok;
        iR = oi;
      }
      any |= __shfl_xor(any, o);
    }
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
      shk[0][w] = kP;
      shi[0][w] = iP;
      shk[1][w] = kR;
      shi[1][w] = iR;
      shany[w] = any;
    }
    __syncthreads();
    kP = shk[0][0];
    iP = shi[0][0];
    kR = shk[1][0];
    iR = shi[1][0];
    any = shany[0];
    for (int v = 1; v < 4; ++v) {
      if (better(shk[0][v], shi[0][v], kP, iP)) {
        kP = shk[0][v];
        iP = shi[0][v];
      }
      if (better(shk[1][v], shi[1][v], kR, iR)) {
        kR = shk[1][v];
        iR = shi[1][v];
      }
      any |= shany[v];
    }
    extra = (rejected && any) ? iR : iP;
  }
  for (int j = threadIdx.x; j <= gam; j += 256) {
    int v;
    if (j < L)
      v = tokens[off + j + 1];
    else if (j == L)
      v = extra;
    else
      v = -1;
    out_tokens[off + j] = v;
  }
  if (threadIdx.x == 0) accept_len[i] = L;
}

void sampler(const StepDesc &d, int B, int M, int V, const float *logits, const int32_t *tokens,
             const float *q, float T, uint64_t seed, float *row_m, float *row_s, int32_t *row_amax,
             int32_t *accept_len, int32_t *out_tokens, hipStream_t s) {
  if (M > 0) row_stats_kernel<<<M, 256, 0, s>>>(logits, V, T, row_m, row_s, row_amax);
  if (B > 0)
    accept_kernel<<<B, 256, 0, s>>>(d, V, logits, tokens, q, T, seed, row_m, row_s, row_amax,
                                    accept_len, out_tokens);
}

__global__ void uniform_kernel(uint64_t seed, uint32_t req, uint32_t tag, uint32_t row, uint32_t n,
                               float *out) {
  for (uint32_t k = blockIdx.x * blockDim.x + threadIdx.x; k < n; k += gridDim.x * blockDim.x)
    out[k] = uniform_from_word(draw(seed, k >> 2, row, req, tag).v[k & 3]);
}

void uniform_draws(uint64_t seed, uint32_t req, uint32_t tag, uint32_t row, uint32_t n, float *out,
                   hipStream_t s) {
  if (n == 0) return;
  uint32_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  uniform_kernel<<<blocks, 256, 0, s>>>(seed, req, tag, row, n, out);
}

__global__ void clear_ints_kernel(int *p, int n) {
  for (int k = blockIdx.x * blockDim.x + threadIdx.x; k < n; k += gridDim.x * blockDim.x) p[k] = 0;
}

void clear_ints(int *p, int n, hipStream_t s) { clear_ints_kernel<<<1, 64, 0, s>>>(p, n); }

}  // namespace wisp
