// Draft-side rejection predictor (Sec. 3.3, Sec. 4.1, App. B): the summary statistics of a draft
// model's next-token distribution (confidence, entropy, top-2 margin, dispersion of the
// logits) and the small MLP that maps them to the probability that the drafted token is
// accepted.  Declared in include/wisp.h.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "../../include/wisp.h"
#include "kernels.h"

namespace wisp {
wisp_status report_error(wisp_status st, const char *msg);
}

namespace {

// The statistics are formed in base 2: y = logits * log2(e) / T, so exp(z - m) = 2^(y - m')
// is one hardware exp2.  A row is cut into chunks of kChunk entries, one workgroup per
// (row, chunk); each thread folds its entries in fp32, each wave merges its lanes in fp32,
// the workgroup merges its waves in fp64, and a second kernel merges the chunks of a row in
// fixed order.  The partial state of a set of entries:
//   m  max y,  s = sum 2^(y - m),  c = sum (y - m) 2^(y - m)  (centred on m: no cancellation
//   against large logits),  v1 >= v2 the two largest y (as a multiset: a repeated maximum
//   gives v2 = v1),  d1 = sum (y - y_0),  d2 = sum (y - y_0)^2 with y_0 the row's first entry.
// Moving the centre from m to m' >= m: s' = r s, c' = r (c + (m - m') s) with r = 2^(m - m').
constexpr int kChunk = 8192;
constexpr float kLog2e = 1.4426950408889634f;

template <typename F>
struct St {
  F m, s, c, v1, v2, d1, d2;
};
using Part = St<double>;

__device__ __forceinline__ void add4(St<float> &a, float4 v, float sc, float y0, int n) {
  float y[4] = {v.x * sc, v.y * sc, v.z * sc, v.w * sc};
  float m4 = y[0];
  for (int k = 1; k < n; ++k) m4 = fmaxf(m4, y[k]);
  if (m4 > a.m) {
    if (a.s > 0.f) {                   // an empty state (m = -inf, s = 0) has nothing to move
      const float r = __builtin_amdgcn_exp2f(a.m - m4);
      a.c = r * fmaf(a.m - m4, a.s, a.c);
      a.s *= r;
    }
    a.m = m4;
  }
  for (int k = 0; k < n; ++k) {
    const float u = y[k] - a.m;
    const float e = __builtin_amdgcn_exp2f(u);
    a.s += e;
    a.c = fmaf(u, e, a.c);
    if (y[k] > a.v1) {
      a.v2 = a.v1;
      a.v1 = y[k];
    } else if (y[k] > a.v2) {
      a.v2 = y[k];
    }
    const float d = y[k] - y0;
    a.d1 += d;
    a.d2 = fmaf(d, d, a.d2);
  }
}

template <typename F>
__device__ __forceinline__ St<F> merge(const St<F> &a, const St<F> &b) {
  St<F> r;
  r.m = a.m > b.m ? a.m : b.m;
  // an empty side (s = 0, m = -inf) contributes nothing: (m - r.m) * s would be -inf * 0
  const F ea = a.s > F(0) ? (F)exp2((double)(a.m - r.m)) : F(0);
  const F eb = b.s > F(0) ? (F)exp2((double)(b.m - r.m)) : F(0);
  r.s = a.s * ea + b.s * eb;
  r.c = (a.s > F(0) ? ea * (a.c + (a.m - r.m) * a.s) : F(0)) + (b.s > F(0) ? eb * (b.c + (b.m - r.m) * b.s) : F(0));
  r.v1 = a.v1 > b.v1 ? a.v1 : b.v1;
  const F lo = a.v1 > b.v1 ? b.v1 : a.v1, hi2 = a.v2 > b.v2 ? a.v2 : b.v2;
  r.v2 = lo > hi2 ? lo : hi2;
  r.d1 = a.d1 + b.d1;
  r.d2 = a.d2 + b.d2;
  return r;
}

// fp32 merge for the in-wave butterfly: the hardware exp2
__device__ __forceinline__ St<float> merge32(const St<float> &a, const St<float> &b) {
  St<float> r;
  r.m = fmaxf(a.m, b.m);
  const float ea = a.s > 0.f ? __builtin_amdgcn_exp2f(a.m - r.m) : 0.f;
  const float eb = b.s > 0.f ? __builtin_amdgcn_exp2f(b.m - r.m) : 0.f;
  r.s = a.s * ea + b.s * eb;
  r.c = (a.s > 0.f ? ea * fmaf(a.m - r.m, a.s, a.c) : 0.f) + (b.s > 0.f ? eb * fmaf(b.m - r.m, b.s, b.c) : 0.f);
  r.v1 = fmaxf(a.v1, b.v1);
  r.v2 = fmaxf(fminf(a.v1, b.v1), fmaxf(a.v2, b.v2));
  r.d1 = a.d1 + b.d1;
  r.d2 = a.d2 + b.d2;
  return r;
}

template <typename F>
__device__ __forceinline__ St<F> shfl(const St<F> &a, int o) {
  return St<F>{__shfl_xor(a.m, o), __shfl_xor(a.s, o), __shfl_xor(a.c, o), __shfl_xor(a.v1, o),
               __shfl_xor(a.v2, o), __shfl_xor(a.d1, o), __shfl_xor(a.d2, o)};
}

__device__ __forceinline__ Part widen(const St<float> &a) {
  return Part{a.m, a.s, a.c, a.v1, a.v2, a.d1, a.d2};
}

// grid (chunks, rows), 256 threads: thread t folds entries 4 (t + 256 k) .. +3 of its chunk
// (16-byte loads) when the row allows them, else entries t + 256 k
__global__ __launch_bounds__(256) void stats_chunk_kernel(const float *__restrict__ logits, int V, int64_t ld,
                                                          float sc, bool vec, Part *__restrict__ parts) {
  const int c = blockIdx.x, nch = gridDim.x;
  const int64_t row = blockIdx.y;
  const float *x = logits + row * ld;
  const float y0 = x[0] * sc;
  St<float> a{-INFINITY, 0.f, 0.f, -INFINITY, -INFINITY, 0.f, 0.f};
  const int base = c * kChunk, end = min(base + kChunk, V);
  if (vec) {
    const float4 *x4 = reinterpret_cast<const float4 *>(x + base);
    float4 buf[kChunk / 1024];
#pragma unroll
    for (int k = 0; k < kChunk / 1024; ++k) {        // all loads of the thread in flight at once
      const int e = (k * 256 + threadIdx.x) * 4;
      buf[k] = base + e + 4 <= end ? x4[k * 256 + threadIdx.x] : float4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int k = 0; k < kChunk / 1024; ++k) {
      const int e = (k * 256 + threadIdx.x) * 4;
      if (base + e + 4 <= end) {
        add4(a, buf[k], sc, y0, 4);
      } else if (base + e < end) {
        float4 v{x[base + e], 0.f, 0.f, 0.f};
        const int n = end - base - e;
        if (n > 1) v.y = x[base + e + 1];
        if (n > 2) v.z = x[base + e + 2];
        add4(a, v, sc, y0, n);
      }
    }
  } else {
    for (int e = base + threadIdx.x; e < end; e += 256) add4(a, float4{x[e], 0.f, 0.f, 0.f}, sc, y0, 1);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) a = merge32(a, shfl(a, o));
  __shared__ Part sh[4];
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = widen(a);
  __syncthreads();
  if (threadIdx.x == 0) parts[row * nch + c] = merge(merge(sh[0], sh[1]), merge(sh[2], sh[3]));
}

// one wave per row: lane l merges chunks l, l + 64, ... in order, then the wave merges (fp64)
__global__ __launch_bounds__(64) void stats_final_kernel(const Part *__restrict__ parts, int nch, int V,
                                                         float4 *__restrict__ stats) {
  const int64_t row = blockIdx.x;
  const int lane = threadIdx.x;
  Part p{-INFINITY, 0.0, 0.0, -INFINITY, -INFINITY, 0.0, 0.0};
  for (int c = lane; c < nch; c += 64) p = merge(p, parts[row * nch + c]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) p = merge(p, shfl(p, o));
  if (lane == 0) {
    const double ln2 = 0.6931471805599453;
    const double p1 = 1.0 / p.s;                       // 2^(v1 - m) = 1
    const double p2 = exp2(p.v2 - p.m) / p.s;          // 0 when V = 1
    const double H = log(p.s) - ln2 * (p.c / p.s);     // -sum p ln p
    const double mean = p.d1 / V;
    const double var = fmax(p.d2 / V - mean * mean, 0.0);
    stats[row] = make_float4((float)p1, (float)H, (float)(p1 - p2), (float)(sqrt(var) * ln2));
  }
}

constexpr int kH1 = 512, kH2 = 128, kH3 = 64;

struct MlpArgs {
  int n_in;
  const float *mean, *inv_std, *w1, *b1, *w2, *b2, *w3, *b3, *w4;
  float b4;
};

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// One workgroup (4 waves) per feature row.  Layers 2 and 3: each wave owns a quarter of the
// outputs; for one output the 64 lanes read a contiguous stretch of its weight row and the
// wave sums their partial dot products in a fixed butterfly order.
__global__ __launch_bounds__(256) void reject_mlp_kernel(MlpArgs p, const float *__restrict__ feat,
                                                         float *__restrict__ prob) {
  __shared__ float x[8], h1[kH1], h2[kH2], h3[kH3];
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid < p.n_in) x[tid] = (feat[(int64_t)row * p.n_in + tid] - p.mean[tid]) * p.inv_std[tid];
  __syncthreads();
  for (int o = tid; o < kH1; o += 256) {
    float acc = p.b1[o];
    for (int k = 0; k < p.n_in; ++k) acc = fmaf(p.w1[o * p.n_in + k], x[k], acc);
    h1[o] = fmaxf(acc, 0.f);
  }
  __syncthreads();
  float hx[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) hx[k] = h1[lane * 8 + k];
  for (int o0 = wave * 32; o0 < wave * 32 + 32; o0 += 4) {    // 512 inputs: 8 per lane, 4 rows in flight
    float4 wv[4][2];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float4 *w = reinterpret_cast<const float4 *>(p.w2 + (int64_t)(o0 + j) * kH1 + lane * 8);
      wv[j][0] = w[0];
      wv[j][1] = w[1];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float w8[8] = {wv[j][0].x, wv[j][0].y, wv[j][0].z, wv[j][0].w,
                           wv[j][1].x, wv[j][1].y, wv[j][1].z, wv[j][1].w};
      float acc = 0.f;
#pragma unroll
      for (int k = 0; k < 8; ++k) acc = fmaf(w8[k], hx[k], acc);
      acc = wave_sum(acc);
      if (lane == 0) h2[o0 + j] = fmaxf(acc + p.b2[o0 + j], 0.f);
    }
  }
  __syncthreads();
  {                                                            // 128 inputs: 2 per lane, 16 rows in flight
    const float ha = h2[lane * 2], hb = h2[lane * 2 + 1];
    float2 wv[16];
#pragma unroll
    for (int j = 0; j < 16; ++j)
      wv[j] = *reinterpret_cast<const float2 *>(p.w3 + (int64_t)(wave * 16 + j) * kH2 + lane * 2);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const float acc = wave_sum(fmaf(wv[j].y, hb, wv[j].x * ha));
      if (lane == 0) h3[wave * 16 + j] = fmaxf(acc + p.b3[wave * 16 + j], 0.f);
    }
  }
  __syncthreads();
  if (wave == 0) {
    const float v = wave_sum(p.w4[lane] * h3[lane]);
    if (lane == 0) prob[row] = 1.f / (1.f + expf(-(v + p.b4)));
  }
}

}  // namespace

using wisp::report_error;

extern "C" size_t wisp_draft_stats_workspace_size(int32_t rows, int32_t vocab) {
  if (rows < 0 || vocab < 1) return 0;
  return (size_t)rows * (size_t)((vocab + kChunk - 1) / kChunk) * sizeof(Part);
}

extern "C" wisp_status wisp_draft_stats(const float *logits, int32_t rows, int32_t vocab, int64_t ld,
                                        float temperature, float *stats, void *workspace, size_t workspace_bytes,
                                        void *stream) {
  if (rows < 0 || vocab < 1 || ld < vocab || !(temperature > 0.f))
    return report_error(WISP_E_INVALID, "wisp_draft_stats: rows < 0, vocab < 1, ld < vocab or temperature <= 0");
  if (rows == 0) return WISP_OK;
  if (rows > 65535) return report_error(WISP_E_UNSUPPORTED, "wisp_draft_stats: more than 65535 rows in one call");
  if (!logits || !stats || !workspace) return report_error(WISP_E_INVALID, "wisp_draft_stats: NULL pointer");
  if (((uintptr_t)stats & 15) != 0 || ((uintptr_t)workspace & 15) != 0)
    return report_error(WISP_E_INVALID, "wisp_draft_stats: stats or workspace not 16-byte aligned");
  if (workspace_bytes < wisp_draft_stats_workspace_size(rows, vocab))
    return report_error(WISP_E_WORKSPACE, "wisp_draft_stats: workspace too small");
  const int nch = (vocab + kChunk - 1) / kChunk;
  const bool vec = ((uintptr_t)logits & 15) == 0 && ld % 4 == 0;
  Part *parts = reinterpret_cast<Part *>(workspace);
  const hipStream_t s = (hipStream_t)stream;
  wisp::launch(stats_chunk_kernel, dim3(nch, rows), dim3(256), 0, s, logits, (int)vocab, (int64_t)ld,
               kLog2e / temperature, vec, parts);
  wisp::launch(stats_final_kernel, dim3(rows), dim3(64), 0, s, (const Part *)parts, nch, (int)vocab,
               reinterpret_cast<float4 *>(stats));
  if (hipGetLastError() != hipSuccess) return report_error(WISP_E_HIP, "wisp_draft_stats: launch failed");
  return WISP_OK;
}

extern "C" wisp_status wisp_reject_predict(const wisp_reject_mlp *mlp, const float *features, int32_t rows,
                                           float *p_accept, void *stream) {
  if (!mlp || rows < 0) return report_error(WISP_E_INVALID, "wisp_reject_predict: NULL mlp or rows < 0");
  if (mlp->n_in < 1 || mlp->n_in > 8) return report_error(WISP_E_INVALID, "wisp_reject_predict: n_in outside 1..8");
  if (rows == 0) return WISP_OK;
  if (!features || !p_accept || !mlp->mean || !mlp->inv_std || !mlp->w1 || !mlp->b1 || !mlp->w2 || !mlp->b2 ||
      !mlp->w3 || !mlp->b3 || !mlp->w4)
    return report_error(WISP_E_INVALID, "wisp_reject_predict: NULL pointer");
  if (((uintptr_t)mlp->w2 & 15) != 0 || ((uintptr_t)mlp->w3 & 7) != 0)
    return report_error(WISP_E_INVALID, "wisp_reject_predict: w2 not 16-byte or w3 not 8-byte aligned");
  MlpArgs a{mlp->n_in, mlp->mean, mlp->inv_std, mlp->w1, mlp->b1, mlp->w2, mlp->b2, mlp->w3, mlp->b3, mlp->w4, mlp->b4};
  wisp::launch(reject_mlp_kernel, dim3(rows), dim3(256), 0, (hipStream_t)stream, a, features, p_accept);
  if (hipGetLastError() != hipSuccess) return report_error(WISP_E_HIP, "wisp_reject_predict: launch failed");
  return WISP_OK;
}
