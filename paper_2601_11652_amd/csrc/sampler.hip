// Acceptance stage of the verification step (Sec. 2.4): Eq. (1) accept draft y_j with
// probability min(1, p/q), Eq. (2) stop at the first rejection R, Eq. (3) emit one extra
// token -- drawn from norm(max(0, p_R - q_R)) after a rejection (the residual that makes
// speculative sampling lossless) and from p after a fully accepted block.
//
// Four launches per batch, over vocabulary chunks of 8192 entries: the row maxima of
// z = logits / T (argmax at T = 0) -- from the LM head's per-tile maxima when the step's own
// GEMM produced them, so the logits are read in full only once more --, the fp64 sums of
// exp(z - max), then one workgroup per
// (request, chunk) decides every draft in parallel (thread j - 1 takes draft j; R is the
// smallest rejected j, an integer minimum) and runs its chunk of the exponential race that
// samples the extra token (argmax of score - ln(-ln u): no prefix sums, so the result does
// not depend on reduction order), and a last kernel combines the chunks' winners in fixed
// order.  All random draws come from Philox4x32-10 keyed by the seed and counted by
// (index, row, request, purpose).
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
// The vocabulary is cut into chunks of kVChunk entries, one workgroup per (row or request,
// chunk).  Partial results are combined in fixed chunk order.
// ---------------------------------------------------------------------------------------
constexpr int kVChunk = 8192;

__device__ __forceinline__ bool better(float ka, int ia, float kb, int ib) {
  return ka > kb || (ka == kb && ia < ib);
}

// (key, index) argmax across the 256 threads; ties go to the smaller index
__device__ __forceinline__ void block_argmax(float &k, int &i, float *shk, int *shi) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ok = __shfl_xor(k, o);
    const int oi = __shfl_xor(i, o);
    if (better(ok, oi, k, i)) {
      k = ok;
      i = oi;
    }
  }
  __syncthreads();
  if ((threadIdx.x & 63) == 0) {
    shk[threadIdx.x >> 6] = k;
    shi[threadIdx.x >> 6] = i;
  }
  __syncthreads();
  k = shk[0];
  i = shi[0];
  for (int w = 1; w < 4; ++w)
    if (better(shk[w], shi[w], k, i)) {
      k = shk[w];
      i = shi[w];
    }
}

// pass 1: per chunk, max of z = l / T (T > 0) or (max, first argmax) of l (T == 0)
__global__ __launch_bounds__(256) void row_max_kernel(const float *__restrict__ logits, int V, float T,
                                                      int CH, float *__restrict__ part_m,
                                                      int32_t *__restrict__ part_i) {
  __shared__ float shk[4];
  __shared__ int shi[4];
  const int c = blockIdx.y;
  const int64_t r = blockIdx.x;
  const float *l = logits + r * V;
  const int k1 = min(V, (c + 1) * kVChunk);
  float bk = -INFINITY;
  int bi = 0x7FFFFFFF;
  for (int k = c * kVChunk + threadIdx.x; k < k1; k += 256) {
    const float z = T == 0.f ? l[k] : l[k] / T;
    if (z > bk) {
      bk = z;
      bi = k;
    }
  }
  block_argmax(bk, bi, shk, shi);
  if (threadIdx.x == 0) {
    part_m[r * CH + c] = bk;
    part_i[r * CH + c] = bi;
  }
}

// pass 1 from the LM head's tile maxima (max and first argmax of the raw logits over each
// output tile): the same values as a pass over the logits.  z = l / T is monotone in l for
// T > 0, so max z = (max l) / T exactly, and the first argmax of l is that of z.  The row's
// result fills all CH chunk slots, so the later passes read it unchanged.
__global__ __launch_bounds__(256) void row_max_from_tiles_kernel(const float *__restrict__ tile_m,
                                                                 const int32_t *__restrict__ tile_i, int tiles,
                                                                 float T, int CH, float *__restrict__ part_m,
                                                                 int32_t *__restrict__ part_i) {
  __shared__ float shk[4];
  __shared__ int shi[4];
  const int64_t r = blockIdx.x;
  float bk = -INFINITY;
  int bi = 0x7FFFFFFF;
  for (int t = threadIdx.x; t < tiles; t += 256) {
    const float v = tile_m[r * tiles + t];
    const int c = tile_i[r * tiles + t];
    if (better(v, c, bk, bi)) {
      bk = v;
      bi = c;
    }
  }
  block_argmax(bk, bi, shk, shi);
  const float m = T == 0.f ? bk : bk / T;
  for (int c = threadIdx.x; c < CH; c += 256) {
    part_m[r * CH + c] = m;
    part_i[r * CH + c] = bi;
  }
}

__device__ __forceinline__ float row_max_of(const float *part_m, int64_t r, int CH) {
  float m = part_m[r * CH];
  for (int c = 1; c < CH; ++c) m = fmaxf(m, part_m[r * CH + c]);
  return m;
}

// pass 2: per chunk, sum of exp(z - m) in fp64 (m = the row's max)
__global__ __launch_bounds__(256) void row_sum_kernel(const float *__restrict__ logits, int V, float T,
                                                      int CH, const float *__restrict__ part_m,
                                                      double *__restrict__ part_s) {
  __shared__ double shd[4];
  const int c = blockIdx.y;
  const int64_t r = blockIdx.x;
  const float *l = logits + r * V;
  const float m = row_max_of(part_m, r, CH);
  const int k1 = min(V, (c + 1) * kVChunk);
  double sum = 0.0;
  for (int k = c * kVChunk + threadIdx.x; k < k1; k += 256) sum += (double)expf(l[k] / T - m);
  sum = block_reduce(sum, shd, [](double a, double b) { return a + b; });
  if (threadIdx.x == 0) part_s[r * CH + c] = sum;
}

struct RowStat {
  float m, S;
  int amax;
};

__device__ RowStat row_stat(const float *part_m, const int32_t *part_i, const double *part_s, int64_t r,
                            int CH, float T) {
  RowStat st;
  if (T == 0.f) {
    float bk = part_m[r * CH];
    int bi = part_i[r * CH];
    for (int c = 1; c < CH; ++c)
      if (better(part_m[r * CH + c], part_i[r * CH + c], bk, bi)) {
        bk = part_m[r * CH + c];
        bi = part_i[r * CH + c];
      }
    st.m = bk;
    st.S = 1.f;
    st.amax = bi;
    return st;
  }
  st.m = row_max_of(part_m, r, CH);
  double s = 0.0;
  for (int c = 0; c < CH; ++c) s += part_s[r * CH + c];
  st.S = (float)s;
  st.amax = -1;
  return st;
}

// pass 3: Eq. (1)-(2) acceptance (recomputed by every chunk's workgroup), then that chunk's
// part of the exponential race for the extra token (Eq. (3) / residual).  The <= 16 draft
// decisions are independent of one another, so thread j - 1 takes draft j's and R is the
// smallest rejected j (gamma + 1 when none is): one round of loads instead of a chain.
__global__ __launch_bounds__(256) void race_kernel(StepDesc d, int V, const float *__restrict__ logits,
                                                   const int32_t *__restrict__ tokens,
                                                   const float *__restrict__ q, float T, uint64_t seed,
                                                   int CH, const float *__restrict__ part_m,
                                                   const int32_t *__restrict__ part_i,
                                                   const double *__restrict__ part_s,
                                                   float *__restrict__ race_k, int32_t *__restrict__ race_i,
                                                   int32_t *__restrict__ req_R) {
  __shared__ int R_sh;
  __shared__ float shk[4];
  __shared__ int shi[4];
  __shared__ int shany[4];
  const int c = blockIdx.y, i = blockIdx.x;
  const int gam = d.gamma[i], off = d.off[i], doff = d.doff[i];
  const uint32_t req = d.req_id[i];
  if (threadIdx.x == 0) R_sh = gam + 1;
  __syncthreads();
  const int j = threadIdx.x + 1;   // gamma <= 16 < 256 threads
  if (j <= gam) {
    int y = tokens[off + j];
    if (y < 0 || y >= V) {
      if (c == 0) flag_error(d.err, kErrToken);
      y = 0;
    }
    const int64_t pr = off + j - 1;
    const RowStat st = row_stat(part_m, part_i, part_s, pr, CH, T);
    bool rejected_j;
    if (T == 0.f) {
      rejected_j = y != st.amax;
    } else {
      const float P = expf(logits[pr * V + y] / T - st.m) / st.S;
      const float Q = q[(int64_t)(doff + j - 1) * V + y];
      const float a = Q > 0.f ? fminf(1.f, P / Q) : (P > 0.f ? 1.f : 0.f);
      const float u = uniform_from_word(draw(seed, 0u, (uint32_t)j, req, kTagAccept).v[0]);
      rejected_j = !(u <= a);
    }
    if (rejected_j) atomicMin(&R_sh, j);   // integer minimum: the order of arrival does not matter
  }
  __syncthreads();
  if (c == 0 && threadIdx.x == 0) req_R[i] = R_sh;
  if (T == 0.f) return;
  const int R = R_sh, r = R - 1;
  const int64_t lr = off + r;
  const float *l = logits + lr * V;
  const bool rejected = R <= gam;
  const float *qr = q + (int64_t)(doff + (rejected ? R - 1 : 0)) * V;
  const RowStat st = row_stat(part_m, part_i, part_s, lr, CH, T);
  float kR = -INFINITY, kP = -INFINITY;
  int iR = 0x7FFFFFFF, iP = 0x7FFFFFFF;
  int any = 0;
  const int k4_0 = c * (kVChunk / 4), k4_1 = min((V + 3) / 4, (c + 1) * (kVChunk / 4));
  for (int k4 = k4_0 + threadIdx.x; k4 < k4_1; k4 += 256) {
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
        const float wk = expf(z - st.m) / st.S - qr[k];
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
  block_argmax(kP, iP, shk, shi);
  block_argmax(kR, iR, shk, shi);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) any |= __shfl_xor(any, o);
  if ((threadIdx.x & 63) == 0) shany[threadIdx.x >> 6] = any;
  __syncthreads();
  if (threadIdx.x == 0) {
    any = shany[0] | shany[1] | shany[2] | shany[3];
    const int64_t o = ((int64_t)i * CH + c) * 2;
    race_k[o] = kP;
    race_i[o] = iP;
    race_k[o + 1] = any ? kR : -INFINITY;
    race_i[o + 1] = any ? iR : 0x7FFFFFFF;
  }
}

// pass 4: combine the chunks' race winners in fixed order, write the outputs
__global__ void finalize_kernel(StepDesc d, int B, const int32_t *__restrict__ tokens, float T, int CH,
                                const float *__restrict__ part_m, const int32_t *__restrict__ part_i,
                                const double *__restrict__ part_s, const float *__restrict__ race_k,
                                const int32_t *__restrict__ race_i, const int32_t *__restrict__ req_R,
                                int32_t *__restrict__ accept_len, int32_t *__restrict__ out_tokens) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B) return;
  const int gam = d.gamma[i], off = d.off[i];
  const int R = req_R[i], L = R - 1;
  int extra;
  if (T == 0.f) {
    extra = row_stat(part_m, part_i, part_s, off + R - 1, CH, T).amax;
  } else {
    float kP = -INFINITY, kR = -INFINITY;
    int iP = 0x7FFFFFFF, iR = 0x7FFFFFFF;
    for (int c = 0; c < CH; ++c) {
      const int64_t o = ((int64_t)i * CH + c) * 2;
      if (better(race_k[o], race_i[o], kP, iP)) {
        kP = race_k[o];
        iP = race_i[o];
      }
      if (race_i[o + 1] != 0x7FFFFFFF && better(race_k[o + 1], race_i[o + 1], kR, iR)) {
        kR = race_k[o + 1];
        iR = race_i[o + 1];
      }
    }
    extra = (R <= gam && iR != 0x7FFFFFFF) ? iR : iP;
  }
  for (int j = 0; j <= gam; ++j) out_tokens[off + j] = j < L ? tokens[off + j + 1] : (j == L ? extra : -1);
  accept_len[i] = L;
}

int sampler_chunks(int V) { return (V + kVChunk - 1) / kVChunk; }

void sampler(const StepDesc &d, int B, int M, int V, const float *logits, const int32_t *tokens,
             const float *q, float T, uint64_t seed, SamplerScratch sc, int32_t *accept_len,
             int32_t *out_tokens, hipStream_t s, RowMaxOut lm) {
  if (B == 0) return;
  const int CH = sampler_chunks(V);
  if (lm.m)
    launch(row_max_from_tiles_kernel, M, 256, 0, s, (const float *)lm.m, (const int32_t *)lm.i, lm.tiles, T, CH,
           sc.part_m, sc.part_i);
  else
    launch(row_max_kernel, dim3(M, CH), 256, 0, s, logits, V, T, CH, sc.part_m, sc.part_i);
  if (T != 0.f) launch(row_sum_kernel, dim3(M, CH), 256, 0, s, logits, V, T, CH, sc.part_m, sc.part_s);
  launch(race_kernel, dim3(B, CH), 256, 0, s, d, V, logits, tokens, q, T, seed, CH, sc.part_m, sc.part_i,
                                          sc.part_s, sc.race_k, sc.race_i, sc.req_R);
  launch(finalize_kernel, (B + 63) / 64, 64, 0, s, d, B, tokens, T, CH, sc.part_m, sc.part_i, sc.part_s,
                                               sc.race_k, sc.race_i, sc.req_R, accept_len, out_tokens);
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
  launch(uniform_kernel, blocks, 256, 0, s, seed, req, tag, row, n, out);
}

__global__ void clear_ints_kernel(int *p, int n) {
  for (int k = blockIdx.x * blockDim.x + threadIdx.x; k < n; k += gridDim.x * blockDim.x) p[k] = 0;
}

void clear_ints(int *p, int n, hipStream_t s) { launch(clear_ints_kernel, 1, 64, 0, s, p, n); }

}  // namespace wisp
