// Ragged multi-query causal attention over the paged KV cache (the attention inside
// Sec. 4.5's batched one-step verification): request i's (gamma_i + 1) * G query rows of
// kv head h attend to keys 0 .. ctx_len_i + j (row j), read page by page through the
// request's block table.
//
// bf16 path, one wave per work item (request, kv head, group of <= 48 query rows, token
// chunk).  Per 32 tokens (two pages) the wave computes S^T = K Q^T and O^T += V^T P^T with
// v_mfma_f32_16x16x32_bf16.  Computing the transposed products keeps every query row in
// one lane column (lane % 16), so the online softmax needs only two cross-lane steps, and
// the probabilities leave the first product in exactly the register order the second one
// consumes (the K index of the PV product is permuted to match, and the V page layout is
// chosen so that permuted operand is two contiguous 8-byte loads per lane).  Chunks of a
// long context are combined afterwards in fixed chunk order.
#include "common.h"
#include "kernels.h"

namespace wisp {

template <int HD, int RB>
__global__ __launch_bounds__(256) void attn_bf16_kernel(StepDesc d, const AttnItem *__restrict__ items,
                                                        int n_items, const uint16_t *__restrict__ q,
                                                        const uint16_t *__restrict__ kp,
                                                        const uint16_t *__restrict__ vp,
                                                        float *__restrict__ part_o,
                                                        float *__restrict__ part_ml, int nq, int nkv,
                                                        float scale) {
  constexpr int KC = HD / 32;   // 32-wide chunks of the QK^T contraction
  constexpr int MB = HD / 16;   // 16-wide blocks of the output head dimension
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int it = blockIdx.x * 4 + wave;
  if (it >= n_items) return;
  const AttnItem item = items[it];
  const int i = item.req, kvh = item.kvh_rbg & 0xFFFF, rbg = item.kvh_rbg >> 16;
  const int G = nq / nkv;
  const int gam = d.gamma[i], ctx = d.ctx[i], off = d.off[i];
  const int rows = (gam + 1) * G;
  const int lr0 = rbg * (16 * RB);
  const int nrb = min(RB, (rows - lr0 + 15) >> 4);
  const int lc = lane & 15, lg = lane >> 4;

  bf16x8_t qf[RB][KC];
  int jrow[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int lr = min(lr0 + rb * 16 + lc, rows - 1);   // padding rows reuse a real row
    jrow[rb] = lr / G;
    const int head = kvh * G + lr % G;
#pragma unroll
    for (int kc = 0; kc < KC; ++kc)
      qf[rb][kc] = as_bf16x8(ld16(q + ((int64_t)(off + jrow[rb]) * nq + head) * HD + kc * 32 + 8 * lg));
  }

  float m_run[RB], l_run[RB];
  floatx4 o[RB][MB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    m_run[rb] = -INFINITY;
    l_run[rb] = 0.f;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) o[rb][mb] = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  const int32_t *pt = d.page_table + (int64_t)i * d.pt_stride;
  const int page_elems = kPage * HD;
  // Block ids of up to 64 pages live in one register (lane l holds page base + l) and are
  // picked with readlane, so a K/V load never waits on a page-table load.
  const int n_pages = (item.t1 + 15) >> 4;
  int pbase = item.t0 >> 4;
  int bids = pt[min(pbase + lane, n_pages - 1)];
  auto block_of = [&](int pg) {
    if (pg >= pbase + 64) {   // wave-uniform: move the window
      pbase = pg;
      bids = pt[min(pbase + lane, n_pages - 1)];
    }
    return __builtin_amdgcn_readlane(bids, pg - pbase);
  };
  // K and V of the page pair starting at token tp.  Block ids are clamped into the pool:
  // tokens past the chunk end get zero probability, and an invalid id is reported.
  auto load_pair = [&](int tp, bf16x8_t (&kf)[2][KC], bf16x8_t (&vf)[MB]) {
    const int pg = tp >> 4;
    const bool has1 = tp + 16 < item.t1;
    int b0 = block_of(pg);
    int b1 = has1 ? block_of(pg + 1) : b0;
    if ((b0 < 0 || b0 >= d.n_blocks || b1 < 0 || b1 >= d.n_blocks) && lane == 0) flag_error(d.err, kErrBlock);
    b0 = min(max(b0, 0), d.n_blocks - 1);
    b1 = min(max(b1, 0), d.n_blocks - 1);
    const uint16_t *K0 = kp + ((int64_t)b0 * nkv + kvh) * page_elems;
    const uint16_t *K1 = kp + ((int64_t)b1 * nkv + kvh) * page_elems;
    const uint16_t *V0 = vp + ((int64_t)b0 * nkv + kvh) * page_elems;
    const uint16_t *V1 = vp + ((int64_t)b1 * nkv + kvh) * page_elems;
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      kf[0][kc] = as_bf16x8(ld16(K0 + kc * 512 + lane * 8));
      kf[1][kc] = as_bf16x8(ld16(K1 + kc * 512 + lane * 8));
    }
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const uint2 a = *reinterpret_cast<const uint2 *>(V0 + mb * 256 + lane * 4);
      const uint2 b = *reinterpret_cast<const uint2 *>(V1 + mb * 256 + lane * 4);
      vf[mb] = as_bf16x8(make_uint4(a.x, a.y, b.x, b.y));
    }
  };
  auto compute_pair = [&](int tp, const bf16x8_t (&kf)[2][KC], const bf16x8_t (&vf)[MB]) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      if (rb >= nrb) break;
      floatx4 s[2];
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        s[p] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kc = 0; kc < KC; ++kc)
          s[p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[p][kc], qf[rb][kc], s[p], 0, 0, 0);
      }
      // s[p][e]: token tp + 16p + 4*lg + e, query row lr0 + rb*16 + lc
      const int lim = min(item.t1, ctx + jrow[rb] + 1);   // causal + chunk end
      float mx = -INFINITY;
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int tok = tp + 16 * p + 4 * lg + e;
          const float v = tok < lim ? s[p][e] * scale : -INFINITY;
          s[p][e] = v;
          mx = fmaxf(mx, v);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run[rb], mx);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = expf(m_run[rb] - m_use);
      float pv[8];
      float rs = 0.f;
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float pr = bf2f(f2bf(expf(s[p][e] - m_use)));   // the value the PV product uses
          pv[p * 4 + e] = pr;
          rs += pr;
        }
      rs += __shfl_xor(rs, 16);
      rs += __shfl_xor(rs, 32);
      l_run[rb] = l_run[rb] * alpha + rs;
      m_run[rb] = m_new;
      const uint4 pw = make_uint4(pack2bf(pv[0], pv[1]), pack2bf(pv[2], pv[3]),
                                  pack2bf(pv[4], pv[5]), pack2bf(pv[6], pv[7]));
      const bf16x8_t pb = as_bf16x8(pw);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        o[rb][mb] *= alpha;
        o[rb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[mb], pb, o[rb][mb], 0, 0, 0);
      }
    }
  };

  // two register sets: the next page pair loads while the current one computes
  bf16x8_t kA[2][KC], vA[MB], kB[2][KC], vB[MB];
  load_pair(item.t0, kA, vA);
  for (int tp = item.t0; tp < item.t1; tp += 64) {
    const bool has2 = tp + 32 < item.t1;
    if (has2) load_pair(tp + 32, kB, vB);
    compute_pair(tp, kA, vA);
    if (!has2) break;
    if (tp + 64 < item.t1) load_pair(tp + 64, kA, vA);
    compute_pair(tp + 32, kB, vB);
  }

  // partials: O [item][hd][64 row slots] (unnormalised), (m, l) [item][64 row slots]
  float *po = part_o + (int64_t)it * HD * 64;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    if (rb >= nrb) break;
    const int rr = rb * 16 + lc;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int e = 0; e < 4; ++e) po[(mb * 16 + 4 * lg + e) * 64 + rr] = o[rb][mb][e];
    if (lg == 0) {
      part_ml[((int64_t)it * 64 + rr) * 2] = m_run[rb];
      part_ml[((int64_t)it * 64 + rr) * 2 + 1] = l_run[rb];
    }
  }
}

// fixed-order combine of a (request, kv head, row group)'s chunks; writes the bf16
// attention output of each (row, q head) into the O-projection's input layout
template <int HD>
__global__ __launch_bounds__(256) void attn_combine_kernel(StepDesc d, const AttnGroup *__restrict__ groups,
                                                           const float *__restrict__ part_o,
                                                           const float *__restrict__ part_ml,
                                                           uint16_t *__restrict__ out, bool packed,
                                                           int out_K, int nq, int nkv) {
  const AttnGroup g = groups[blockIdx.x];
  const int G = nq / nkv;
  const int rows = (d.gamma[g.req] + 1) * G;
  const int lr0 = g.rbg * kAttnRowsPerItem;
  const int nr = min(kAttnRowsPerItem, rows - lr0);
  const int off = d.off[g.req];
  constexpr int CH = HD / 8;
  for (int u = threadIdx.x; u < nr * CH; u += 256) {
    const int rr = u % nr, c0 = (u / nr) * 8;   // neighbouring lanes read neighbouring rows
    float m = -INFINITY;
    for (int c = 0; c < g.n_items; ++c) m = fmaxf(m, part_ml[((int64_t)(g.first_item + c) * 64 + rr) * 2]);
    float den = 0.f;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < g.n_items; ++c) {
      const int64_t itm = g.first_item + c;
      const float mc = part_ml[(itm * 64 + rr) * 2];
      if (mc == -INFINITY) continue;
      const float w = expf(mc - m);
      den += part_ml[(itm * 64 + rr) * 2 + 1] * w;
      const float *po = part_o + itm * HD * 64;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += po[(c0 + e) * 64 + rr] * w;
    }
    const int lr = lr0 + rr;
    const int64_t row = off + lr / G;
    const int head = g.kvh * G + lr % G;
    const int64_t col = (int64_t)head * HD + c0;
    uint4 w4;
    const float inv = 1.0f / den;
    w4.x = pack2bf(acc[0] * inv, acc[1] * inv);
    w4.y = pack2bf(acc[2] * inv, acc[3] * inv);
    w4.z = pack2bf(acc[4] * inv, acc[5] * inv);
    w4.w = pack2bf(acc[6] * inv, acc[7] * inv);
    const int64_t o = packed ? packed_off(row, col, out_K) : row * out_K + col;
    *reinterpret_cast<uint4 *>(out + o) = w4;
  }
}

void attention_bf16_main(const StepDesc &d, const AttnItem *items, int n_items, const uint16_t *q,
                         const uint16_t *k_pool, const uint16_t *v_pool, float *part_o, float *part_ml,
                         int nq, int nkv, int hd, hipStream_t s) {
  if (n_items == 0) return;
  const float scale = 1.0f / sqrtf((float)hd);
  const int blocks = (n_items + 3) / 4;
  constexpr int RB = kAttnRowsPerItem / 16;
  if (hd == 128)
    attn_bf16_kernel<128, RB><<<blocks, 256, 0, s>>>(d, items, n_items, q, k_pool, v_pool, part_o, part_ml, nq, nkv, scale);
  else
    attn_bf16_kernel<64, RB><<<blocks, 256, 0, s>>>(d, items, n_items, q, k_pool, v_pool, part_o, part_ml, nq, nkv, scale);
}

void attention_bf16_combine(const StepDesc &d, const AttnGroup *groups, int n_groups,
                            const float *part_o, const float *part_ml, uint16_t *out, bool out_packed,
                            int out_K, int nq, int nkv, int hd, hipStream_t s) {
  if (n_groups == 0) return;
  if (hd == 128)
    attn_combine_kernel<128><<<n_groups, 256, 0, s>>>(d, groups, part_o, part_ml, out, out_packed, out_K, nq, nkv);
  else
    attn_combine_kernel<64><<<n_groups, 256, 0, s>>>(d, groups, part_o, part_ml, out, out_packed, out_K, nq, nkv);
}

// ---------------------------------------------------------------------------------------
// fp32 path (small models): one workgroup per (request, q head), plain VALU
// ---------------------------------------------------------------------------------------
__device__ __forceinline__ float block_reduce_256(float v, float *sh, bool is_max) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float w = __shfl_xor(v, o);
    v = is_max ? fmaxf(v, w) : v + w;
  }
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  return is_max ? fmaxf(fmaxf(sh[0], sh[1]), fmaxf(sh[2], sh[3])) : sh[0] + sh[1] + sh[2] + sh[3];
}

__global__ __launch_bounds__(256) void attn_f32_kernel(StepDesc d, const float *__restrict__ q,
                                                       const float *__restrict__ kp,
                                                       const float *__restrict__ vp,
                                                       float *__restrict__ out, int nq, int nkv, int hd,
                                                       float scale) {
  extern __shared__ float sc[];
  __shared__ float sh[4];
  const int i = blockIdx.x / nq, hq = blockIdx.x % nq;
  const int kvh = hq / (nq / nkv);
  const int gam = d.gamma[i], ctx = d.ctx[i], off = d.off[i];
  const int32_t *pt = d.page_table + (int64_t)i * d.pt_stride;
  const int page_elems = kPage * hd;
  for (int j = 0; j <= gam; ++j) {
    const int64_t r = off + j;
    const float *qr = q + (r * nq + hq) * hd;
    const int T = ctx + j + 1;
    float mx = -INFINITY;
    for (int t = threadIdx.x; t < T; t += 256) {
      const int blk = pt[t / kPage];
      float dot = 0.f;
      if (blk >= 0 && blk < d.n_blocks) {
        const float *pg = kp + ((int64_t)blk * nkv + kvh) * page_elems;
        for (int e = 0; e < hd; ++e) dot += qr[e] * pg[k_page_off(t % kPage, e)];
      } else {
        flag_error(d.err, kErrBlock);
      }
      sc[t] = dot * scale;
      mx = fmaxf(mx, sc[t]);
    }
    mx = block_reduce_256(mx, sh, true);
    float sum = 0.f;
    for (int t = threadIdx.x; t < T; t += 256) {
      const float p = expf(sc[t] - mx);
      sc[t] = p;
      sum += p;
    }
    sum = block_reduce_256(sum, sh, false);
    __syncthreads();
    for (int e = threadIdx.x; e < hd; e += 256) {
      float acc = 0.f;
      for (int t = 0; t < T; ++t) {
        const int blk = pt[t / kPage];
        if (blk < 0 || blk >= d.n_blocks) continue;
        acc += sc[t] * vp[((int64_t)blk * nkv + kvh) * page_elems + v_page_off(t % kPage, e)];
      }
      out[(r * nq + hq) * hd + e] = acc / sum;
    }
    __syncthreads();
  }
}

void attention_f32(const StepDesc &d, int B, const float *q, const float *k_pool,
                   const float *v_pool, float *out, int nq, int nkv, int hd, int max_tokens,
                   hipStream_t s) {
  const float scale = 1.0f / sqrtf((float)hd);
  attn_f32_kernel<<<B * nq, 256, max_tokens * sizeof(float), s>>>(d, q, k_pool, v_pool, out, nq, nkv, hd, scale);
}

}  // namespace wisp
