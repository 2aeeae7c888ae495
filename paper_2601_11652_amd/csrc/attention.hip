// Ragged multi-query causal attention over the paged KV cache (the attention inside
// Sec. 4.5's batched one-step verification): request i's (gamma_i + 1) * G query rows of
// kv head h attend to keys 0 .. ctx_len_i + j (row j), read page by page through the
// request's block table.
//
// bf16 path, one wave per work item (request, kv head, group of <= 48 query rows, token
// chunk).  Per 32 tokens (a page pair) the wave computes S^T = K Q^T and O^T += V^T P^T
// with v_mfma_f32_16x16x32_bf16.  Computing the transposed products keeps every query row
// in one lane column (lane % 16), so the online softmax needs only two cross-row steps
// (VALU lane swaps),
// and the probabilities leave the first product in exactly the register order the second
// one consumes.  The token order inside the pair is chosen (through the K and V page
// layouts) so that lane group g = lane / 16 holds tokens 8g .. 8g + 7 of the pair, all in
// one page: the V operand of each lane is then one 16-byte load, and the K operand of
// each product row one 16-byte load.  Chunks of a long context are combined afterwards in
// fixed chunk order.
#include "common.h"
#include "kernels.h"

namespace wisp {

template <int HD, int RB, int NB>
__global__ __launch_bounds__(256) void attn_bf16_kernel(StepDesc d, const AttnItem *__restrict__ items,
                                                        int n_items, const uint16_t *__restrict__ q,
                                                        const uint16_t *__restrict__ kp,
                                                        const uint16_t *__restrict__ vp,
                                                        float *__restrict__ part_o,
                                                        float *__restrict__ part_ml, int nq, int nkv,
                                                        float scale) {
  constexpr int KC = HD / 32;   // 32-wide chunks of the QK^T contraction
  constexpr int MB = HD / 16;   // 16-wide blocks of the output head dimension
  // the work item is wave-uniform: keeping it in scalar registers makes every branch and
  // loop bound below scalar, so the loads of the next page pair stay in flight while the
  // current pair is computed (with vector-held bounds the waits collapse to "all loads")
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int it = blockIdx.x * 4 + wave;
  if (it >= n_items) return;
  AttnItem item;
  item.req = __builtin_amdgcn_readfirstlane(items[it].req);
  item.kvh_rbg = __builtin_amdgcn_readfirstlane(items[it].kvh_rbg);
  item.t0 = __builtin_amdgcn_readfirstlane(items[it].t0);
  item.t1 = __builtin_amdgcn_readfirstlane(items[it].t1);
  const int i = item.req, kvh = item.kvh_rbg & 0xFFFF, rbg = item.kvh_rbg >> 16;
  const int G = nq / nkv;
  const int nrw = __builtin_amdgcn_readfirstlane(d.nrow[i]);
  const int ctx = __builtin_amdgcn_readfirstlane(d.ctx[i]);
  const int off = __builtin_amdgcn_readfirstlane(d.off[i]);
  const int rows = nrw * G;
  const int lr0 = rbg * (16 * RB);
  // row blocks this wave carries: at least one (an item always has rows), written so the
  // compiler can see it and never skips a pair's products (a skipped product would leave
  // its loads pending across the loop)
  const int nrb = 1 + max(0, min(RB - 1, (rows - lr0 - 1) >> 4));
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
  // The item's block ids (at most 64 pages) live in one register, lane l holding page
  // t0 / 16 + l, and are picked with readlane: no page-table load inside the loop, so no
  // wait in it covers more than the pair being consumed.
  const int pbase = item.t0 >> 4;
  const int n_pages = (item.t1 + 15) >> 4;
  const int bids = pt[min(pbase + lane, n_pages - 1)];
  auto block_of = [&](int pg) { return __builtin_amdgcn_readlane(bids, pg - pbase); };
  // Per-lane operand offsets inside a page.  Row r = lane % 16 of the S product for page
  // half h (0/1) is token 16 * (r / 8) + 8 * ((r / 4) % 2) + 4 * h + r % 4 of the pair;
  // lane group g then holds probabilities of tokens 8g .. 8g + 7, which sit in page g / 2.
  const int k_off = lg * 64 + (lc & 7) * 8;           // + (kc * 2 + h) * 256
  const int v_off = (lg & 1) * 128 + lc * 8;          // + mb * 256
  const bool k_hi = lc >= 8, v_hi = lg >= 2;           // which page of the pair
  // K and V of the page pair starting at token tp.  Block ids are clamped into the pool:
  // tokens past the chunk end get zero probability, and an invalid id is reported.
  auto load_pair = [&](int tp, bf16x8_t (&kf)[2][KC], bf16x8_t (&vf)[MB]) {
    const int pg = tp >> 4;
    int b0 = block_of(pg);
    int b1 = tp + 16 < item.t1 ? block_of(pg + 1) : b0;
    if ((b0 < 0 || b0 >= d.n_blocks || b1 < 0 || b1 >= d.n_blocks) && lane == 0) flag_error(d.err, kErrBlock);
    b0 = min(max(b0, 0), d.n_blocks - 1);
    b1 = min(max(b1, 0), d.n_blocks - 1);
    const int64_t kv0 = ((int64_t)b0 * nkv + kvh) * page_elems;
    const int64_t kv1 = ((int64_t)b1 * nkv + kvh) * page_elems;
    const uint16_t *K = kp + (k_hi ? kv1 : kv0) + k_off;
    const uint16_t *V = vp + (v_hi ? kv1 : kv0) + v_off;
    // every K and V byte is read once per step: non-temporal, so the stream does not evict
    // the attention partials that the combine kernel reads next (measured: the combine runs
    // about a third faster at long contexts, the attention itself about 5 % faster)
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      kf[0][kc] = as_bf16x8(ld16_stream(K + (kc * 2) * 256));
      kf[1][kc] = as_bf16x8(ld16_stream(K + (kc * 2 + 1) * 256));
    }
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) vf[mb] = as_bf16x8(ld16_stream(V + mb * 256));
  };
  // Online softmax in the raw score domain: p = 2^((s - m) * c) with c = scale * log2(e),
  // one FMA and one v_exp per score.  The running maximum m of a row is raised only when
  // a score exceeds it by more than kTau / c (p then stays below 2^kTau), so the O
  // accumulators are rescaled only on the rare pairs that raise some row's maximum; the
  // result is unchanged because numerator and denominator share the same reference.
  const float c_log2 = scale * 1.4426950408889634f;
  constexpr float kTau = 8.0f;
  const float tau_raw = kTau / c_log2;
  auto compute_pair = [&](int tp, const bf16x8_t (&kf)[2][KC], const bf16x8_t (&vf)[MB]) {
    // scalar: no token of this pair lies past the chunk end or any row's causal limit
    const bool unmasked = tp + 32 <= min(item.t1, ctx + 1);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      if (rb >= nrb) break;
      floatx4 s[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        s[h] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kc = 0; kc < KC; ++kc)
          s[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[h][kc], qf[rb][kc], s[h], 0, 0, 0);
      }
      // s[h][e]: token tp + 8 * lg + 4 * h + e, query row lr0 + rb*16 + lc
      if (!unmasked) {
        const int lim = min(item.t1, ctx + jrow[rb] + 1);   // causal + chunk end
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (tp + 8 * lg + 4 * h + e >= lim) s[h][e] = -INFINITY;
      }
      float mx = fmaxf(fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3])),
                       fmaxf(fmaxf(s[1][0], s[1][1]), fmaxf(s[1][2], s[1][3])));
      mx = xor32_max(xor16_max(mx));
      const bool grow = mx > m_run[rb] + tau_raw;   // false while the row has seen no token
      if (__builtin_amdgcn_ballot_w64(grow)) {      // wave-uniform: some row raises its max
        const float alpha = grow ? __builtin_amdgcn_exp2f((m_run[rb] - mx) * c_log2) : 1.0f;
        m_run[rb] = grow ? mx : m_run[rb];
        l_run[rb] *= alpha;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) o[rb][mb] *= alpha;
      }
      const float mc = m_run[rb] == -INFINITY ? 0.f : m_run[rb] * c_log2;
      // probabilities rounded to bf16 once; the row sum adds exactly the rounded values
      uint32_t pw[4];
      float rs = 0.f;
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int e = 0; e < 4; e += 2) {
          const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[h][e], c_log2, -mc));
          const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[h][e + 1], c_log2, -mc));
          const uint32_t pk = pack2bf_rne(p0, p1);
          pw[h * 2 + e / 2] = pk;
          rs += __uint_as_float(pk << 16) + __uint_as_float(pk & 0xFFFF0000u);
        }
      rs = xor32_sum(xor16_sum(rs));
      l_run[rb] += rs;
      const bf16x8_t pb = as_bf16x8(make_uint4(pw[0], pw[1], pw[2], pw[3]));
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
        o[rb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[mb], pb, o[rb][mb], 0, 0, 0);
    }
  };

  // A ring of NB register sets: while one pair is computed, the next NB - 1 pairs load.
  // The loop body is unrolled over the ring (static register indices), has a single exit
  // at the bottom, and issues every load unconditionally (a pair index past the end
  // re-reads the last pair, a cache hit), so each wait covers exactly the pair being
  // consumed while the others stay in flight.
  const int np = (item.t1 - item.t0 + 31) >> 5;
  auto pair_t = [&](int k) { return item.t0 + 32 * min(k, np - 1); };
  bf16x8_t kr[NB][2][KC], vr[NB][MB];
#pragma unroll
  for (int b = 0; b + 1 < NB; ++b) load_pair(pair_t(b), kr[b], vr[b]);
  int k = 0;
  for (; k + NB <= np; k += NB) {
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      load_pair(pair_t(k + b + NB - 1), kr[(b + NB - 1) % NB], vr[(b + NB - 1) % NB]);
      __builtin_amdgcn_sched_barrier(0);
      compute_pair(item.t0 + 32 * (k + b), kr[b], vr[b]);
    }
  }
#pragma unroll
  for (int b = 0; b + 1 < NB; ++b)
    if (k + b < np) compute_pair(item.t0 + 32 * (k + b), kr[b], vr[b]);

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
      // m in the scaled natural-log domain: chunk weights are exp(m_chunk - m_max)
      part_ml[((int64_t)it * 64 + rr) * 2] = m_run[rb] == -INFINITY ? -INFINITY : m_run[rb] * scale;
      part_ml[((int64_t)it * 64 + rr) * 2 + 1] = l_run[rb];
    }
  }

}

// Fixed-order combine of each group's chunk partials: one thread per (row, 8 head dims).
// Pass 1 takes the maximum of the chunks' running maxima, pass 2 adds the rescaled chunk
// sums in chunk order.  A group of at most MAXC chunks loads everything in one round; a
// longer one loads its maxima 2 MAXC at a time and keeps two rounds of MAXC chunks in
// flight in pass 2 (B = 4, 22 chunks per group: 14.6 -> 10.2 us per launch).
// Writes the bf16 attention output of each (row, q head) into the O-projection's input
// layout.
template <int HD, int MAXC, bool LONG>
__global__ __launch_bounds__(256) void attn_combine_kernel(StepDesc d, const AttnGroup *__restrict__ groups,
                                                           int n_groups, const float *__restrict__ part_o,
                                                           const float *__restrict__ part_ml,
                                                           uint16_t *__restrict__ out, bool packed, int out_K,
                                                           int nq, int nkv) {
  constexpr int CH = HD / 8;
  constexpr int UNITS = kAttnRowsPerItem * CH;   // (row slot, 8-dim chunk) pairs per group
  const int64_t u_all = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int gi = (int)(u_all / UNITS);
  if (gi >= n_groups) return;
  const AttnGroup g = groups[gi];
  const int G = nq / nkv;
  const int rows = d.nrow[g.req] * G;
  const int lr0 = g.rbg * kAttnRowsPerItem;
  const int nr = min(kAttnRowsPerItem, rows - lr0);
  const int u = (int)(u_all % UNITS);
  const int rr = u % kAttnRowsPerItem, c0 = (u / kAttnRowsPerItem) * 8;   // neighbouring threads: rows
  if (rr >= nr) return;
  const int n = g.n_items;
  auto item_of = [&](int c) { return (int64_t)g.first_item + min(c, n - 1); };   // clamped, in range

  // a group's threads fill whole waves (UNITS is a multiple of 64), so `cb + c < n` is
  // wave-uniform: chunks past the group's last are not loaded at all
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float den = 0.f;
  float m = -INFINITY;
  if (!LONG || n <= MAXC) {
    // at most MAXC chunks (every group, where the host launches the short instance): one
    // round of loads: every chunk's (m, l) and O values at once, the maximum taken from
    // registers; the same sums in the same order as the two-pass form below
    float mc[MAXC], lc[MAXC], pv[MAXC][8];
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
      mc[c] = -INFINITY;
      lc[c] = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) pv[c][e] = 0.f;
      if (c < n) {
        const int64_t itm = item_of(c);
        mc[c] = part_ml[(itm * 64 + rr) * 2];
        lc[c] = part_ml[(itm * 64 + rr) * 2 + 1];
        const float *po = part_o + (itm * HD + c0) * 64 + rr;
#pragma unroll
        for (int e = 0; e < 8; ++e) pv[c][e] = po[e * 64];
      }
    }
#pragma unroll
    for (int c = 0; c < MAXC; ++c)
      if (c < n) m = fmaxf(m, mc[c]);
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
      if (c >= n || mc[c] == -INFINITY) continue;
      const float w = expf(mc[c] - m);
      den += lc[c] * w;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += pv[c][e] * w;
    }
  } else {
    // a longer group (the long instance, launched when some group has more than MAXC
    // chunks; the branch is wave-uniform, since a group fills whole waves)
    // pass 1: the group's maximum, 2 MAXC chunks' m per round, all loaded before any is used
    constexpr int MC1 = 2 * MAXC;
    for (int cb = 0; cb < n; cb += MC1) {
      float mc[MC1];
#pragma unroll
      for (int c = 0; c < MC1; ++c) mc[c] = part_ml[(item_of(cb + c) * 64 + rr) * 2];
#pragma unroll
      for (int c = 0; c < MC1; ++c) m = cb + c < n ? fmaxf(m, mc[c]) : m;
    }
    // pass 2: the rescaled sums in chunk order, in rounds of R = MAXC / 2 chunks with the
    // next round's loads issued before the current round is used (MAXC chunks in flight in
    // the registers of one MAXC round).  The loads are unconditional (clamped to the
    // group's last chunk) and chunks past it are dropped by selects, so no branch separates
    // a load from its use and the waits stay exact.
    constexpr int R = MAXC / 2;
    float mc0[R], lc0[R], pv0[R][8], mc1[R], lc1[R], pv1[R][8];
    auto load = [&](float (&mc)[R], float (&lc)[R], float (&pv)[R][8], int cb) {
#pragma unroll
      for (int c = 0; c < R; ++c) {
        const int64_t itm = item_of(cb + c);
        mc[c] = part_ml[(itm * 64 + rr) * 2];
        lc[c] = part_ml[(itm * 64 + rr) * 2 + 1];
        const float *po = part_o + (itm * HD + c0) * 64 + rr;
#pragma unroll
        for (int e = 0; e < 8; ++e) pv[c][e] = po[e * 64];
      }
    };
    auto use = [&](const float (&mc)[R], const float (&lc)[R], const float (&pv)[R][8], int cb) {
#pragma unroll
      for (int c = 0; c < R; ++c) {
        const bool ok = cb + c < n && mc[c] != -INFINITY;
        const float w = expf(mc[c] - m);
        den = ok ? den + lc[c] * w : den;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = ok ? acc[e] + pv[c][e] * w : acc[e];
      }
    };
    load(mc0, lc0, pv0, 0);
    for (int cb = 0; cb < n; cb += 2 * R) {
      load(mc1, lc1, pv1, cb + R);
      use(mc0, lc0, pv0, cb);
      load(mc0, lc0, pv0, cb + 2 * R);
      use(mc1, lc1, pv1, cb + R);
    }
  }
  const int lr = lr0 + rr;
  const int64_t row = d.off[g.req] + lr / G;
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

void attention_bf16_main(const StepDesc &d, const AttnItem *items, int n_items, const uint16_t *q,
                         const uint16_t *k_pool, const uint16_t *v_pool, float *part_o, float *part_ml,
                         int nq, int nkv, int hd, hipStream_t s) {
  if (n_items == 0) return;
  const float scale = 1.0f / sqrtf((float)hd);
  const int blocks = (n_items + 3) / 4;
  constexpr int RB = kAttnRowsPerItem / 16;
  constexpr int kAttnRing = 2;   // page pairs in registers: one computed, one loading
  if (hd == 128)
    launch(attn_bf16_kernel<128, RB, kAttnRing>, blocks, 256, 0, s, d, items, n_items, q, k_pool, v_pool, part_o, part_ml, nq, nkv, scale);
  else
    launch(attn_bf16_kernel<64, RB, kAttnRing>, blocks, 256, 0, s, d, items, n_items, q, k_pool, v_pool, part_o, part_ml, nq, nkv, scale);
}

void attention_bf16_combine(const StepDesc &d, const AttnGroup *groups, int n_groups, int max_group_chunks,
                            const float *part_o, const float *part_ml, uint16_t *out, bool out_packed,
                            int out_K, int nq, int nkv, int hd, hipStream_t s) {
  if (n_groups == 0) return;
  constexpr int kMaxC = kAttnCombineChunks;
  const bool longer = max_group_chunks > kMaxC;
  const int64_t threads = (int64_t)n_groups * kAttnRowsPerItem * (hd / 8);
  const unsigned blocks = (unsigned)((threads + 255) / 256);
  if (hd == 128)
    launch(longer ? attn_combine_kernel<128, kMaxC, true> : attn_combine_kernel<128, kMaxC, false>, blocks, 256, 0,
           s, d, groups, n_groups, part_o, part_ml, out, out_packed, out_K, nq, nkv);
  else
    launch(longer ? attn_combine_kernel<64, kMaxC, true> : attn_combine_kernel<64, kMaxC, false>, blocks, 256, 0, s,
           d, groups, n_groups, part_o, part_ml, out, out_packed, out_K, nq, nkv);
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
  const int nrw = d.nrow[i], ctx = d.ctx[i], off = d.off[i];
  const int32_t *pt = d.page_table + (int64_t)i * d.pt_stride;
  const int page_elems = kPage * hd;
  for (int j = 0; j < nrw; ++j) {
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
  launch(attn_f32_kernel, B * nq, 256, max_tokens * sizeof(float), s, d, q, k_pool, v_pool, out, nq, nkv, hd, scale);
}

}  // namespace wisp
