// C ABI of the verification step (declared in include/wisp.h): validation, planning of
// the launch (row layout, GEMM K-splits, split-KV attention work list), workspace carving
// and the stream-ordered kernel sequence of one step.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/wisp.h"
#include "common.h"
#include "host_guard.h"
#include "kernels.h"

using namespace wisp;

namespace {

// the calling thread's last error message (a fixed buffer: reporting never allocates)
thread_local char g_last_error[512] = "";

wisp_status fail(wisp_status st, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
wisp_status fail(wisp_status st, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// ------------------------------------------------------------------------------------------
// launch plan
// ------------------------------------------------------------------------------------------
struct Plan {
  int B = 0, M = 0, Mp = 0, S = 0;   // requests, rows, rows padded to 32, total drafts
  int Mv = 0;                        // verification rows (root and drafts): logits rows
  bool prefill = false;              // some request forwards prompt rows before its root
  int d = 0, nq = 0, nkv = 0, hd = 0, F = 0, V = 0, qdim = 0, kvdim = 0, qkvN = 0, G = 0;
  bool bf16 = false;
  int max_tokens = 0;
  GemmCfg g_qkv{}, g_o{}, g_gu{}, g_down{}, g_lm{};
  std::vector<AttnItem> items;
  std::vector<AttnGroup> groups;
  std::vector<int32_t> host;         // descriptor block uploaded to the device
  // int32 offsets inside the descriptor block
  size_t i_off = 0, i_doff = 0, i_gamma = 0, i_ctx = 0, i_req = 0, i_row_req = 0, i_row_pos = 0,
         i_items = 0, i_groups = 0, i_voff = 0, i_nrow = 0, i_vrow = 0;
  // byte offsets inside the workspace
  size_t w_err = 0, w_desc = 0, w_rope = 0, w_h = 0, w_xn = 0, w_ao = 0, w_af = 0, w_q = 0,
         w_part = 0, w_attn_o = 0, w_attn_ml = 0, w_sm = 0, w_si = 0, w_ss = 0, w_rk = 0, w_ri = 0,
         w_rR = 0, w_vtok = 0, w_lmm = 0, w_lmi = 0, total = 0;
  int lm_tiles = 0;                  // output tiles of the LM head (bf16): its row-maxima columns
  int max_group_chunks = 0;          // most chunks any attention group combines
};


wisp_status check_model(const wisp_model *m, bool need_weights) {
  if (!m) return fail(WISP_E_INVALID, "model is NULL");
  if (m->n_layers <= 0 || m->d_model <= 0 || m->n_q_heads <= 0 || m->n_kv_heads <= 0 ||
      m->head_dim <= 0 || m->d_ff <= 0 || m->vocab <= 0)
    return fail(WISP_E_INVALID, "model dimensions must be positive");
  if (m->dtype != WISP_F32 && m->dtype != WISP_BF16) return fail(WISP_E_UNSUPPORTED, "dtype %d", m->dtype);
  if (m->n_q_heads % m->n_kv_heads) return fail(WISP_E_UNSUPPORTED, "n_q_heads %% n_kv_heads != 0");
  if (m->head_dim % 32 || m->head_dim > 256)
    return fail(WISP_E_UNSUPPORTED, "head_dim must be a multiple of 32, at most 256");
  if (m->d_model % 32 || m->d_ff % 32) return fail(WISP_E_UNSUPPORTED, "d_model, d_ff must be multiples of 32");
  // the residual + norm kernels hold a row in one workgroup, 8 columns per thread
  if (m->d_model > 8192) return fail(WISP_E_UNSUPPORTED, "d_model > 8192");
  if (m->dtype == WISP_BF16) {
    if (m->head_dim != 64 && m->head_dim != 128) return fail(WISP_E_UNSUPPORTED, "bf16 head_dim must be 64 or 128");
    if (m->vocab % 32) return fail(WISP_E_UNSUPPORTED, "bf16 vocab must be a multiple of 32");
    if (m->n_q_heads / m->n_kv_heads > 64) return fail(WISP_E_UNSUPPORTED, "GQA group > 64");
  }
  if (!(m->rms_eps >= 0.f) || !(m->rope_base > 0.f)) return fail(WISP_E_INVALID, "rms_eps / rope_base");
  if (need_weights) {
    if (!m->embed || !m->final_norm || !m->lm_head || !m->attn_norm || !m->w_qkv || !m->w_o ||
        !m->mlp_norm || !m->w_gate_up || !m->w_down)
      return fail(WISP_E_INVALID, "NULL weight pointer");
    for (int l = 0; l < m->n_layers; ++l)
      if (!m->attn_norm[l] || !m->w_qkv[l] || !m->w_o[l] || !m->mlp_norm[l] || !m->w_gate_up[l] ||
          !m->w_down[l])
        return fail(WISP_E_INVALID, "NULL weight pointer in layer %d", l);
  }
  return WISP_OK;
}

// forward: the call runs the model, so prompt rows count towards the batch's rows
wisp_status check_desc(const wisp_batch_desc *d, bool need_pages, bool forward) {
  if (!d) return fail(WISP_E_INVALID, "batch descriptor is NULL");
  if (d->B < 0) return fail(WISP_E_INVALID, "B < 0");
  if (d->B == 0) return WISP_OK;
  if (!d->ctx_len || !d->gamma) return fail(WISP_E_INVALID, "ctx_len / gamma is NULL");
  if (!(d->temperature >= 0.f) || std::isinf(d->temperature)) return fail(WISP_E_INVALID, "temperature must be finite and >= 0");
  int64_t rows = 0;
  for (int i = 0; i < d->B; ++i) {
    if (d->gamma[i] < 0 || d->gamma[i] > WISP_GAMMA_MAX)
      return fail(WISP_E_INVALID, "gamma[%d] = %d outside 0..%d", i, d->gamma[i], WISP_GAMMA_MAX);
    if (d->ctx_len[i] < 0) return fail(WISP_E_INVALID, "ctx_len[%d] < 0", i);
    const int pre = d->prefill_len ? d->prefill_len[i] : 0;
    if (pre < 0 || pre > WISP_PREFILL_MAX)
      return fail(WISP_E_INVALID, "prefill_len[%d] = %d outside 0..%d", i, pre, WISP_PREFILL_MAX);
    const int64_t need = (int64_t)d->ctx_len[i] + pre + d->gamma[i] + 1;
    if (need > INT32_MAX / 2) return fail(WISP_E_INVALID, "request %d: ctx_len too large", i);
    if (need_pages && (int64_t)d->pt_stride * WISP_PAGE < need)
      return fail(WISP_E_CAPACITY, "request %d needs %lld tokens but the page table holds %d", i,
                  (long long)need, d->pt_stride * WISP_PAGE);
    // the model's rows are bounded by WISP_ROWS_MAX; the acceptance alone only by int range
    rows += (forward ? pre : 0) + d->gamma[i] + 1;
    const int64_t max_rows = forward ? WISP_ROWS_MAX : kAcceptRowsMax;
    if (rows > max_rows)
      return fail(WISP_E_UNSUPPORTED, "the batch has more than %lld rows (prompt, root and draft rows)",
                  (long long)max_rows);
  }
  if (need_pages && !d->kv_page_table) return fail(WISP_E_INVALID, "kv_page_table is NULL");
  return WISP_OK;
}

void carve(size_t &w, size_t &field, size_t bytes) {
  field = w;
  w = align256(w + bytes);
}

// forward=true: the full step; false: acceptance only (rows/drafts of the batch, vocab V)
// compute units of the current device (the attention work list is sized to them)
int device_cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    n = 256;
  return n;
}

wisp_status make_plan(Plan &p, const wisp_model *m, const wisp_batch_desc *d, bool forward, int vocab = 0) {
  p.B = d->B;
  p.V = forward ? m->vocab : vocab;
  // rows of request i: prefill_len prompt rows (forward only), root, gamma drafts; the
  // verification rows (root .. y_gamma) are the last gamma + 1 and alone produce logits
  std::vector<int> off(p.B + 1, 0), doff(p.B + 1, 0), voff(p.B + 1, 0), nrow(p.B, 0);
  for (int i = 0; i < p.B; ++i) {
    const int pre = (forward && d->prefill_len) ? d->prefill_len[i] : 0;
    nrow[i] = pre + d->gamma[i] + 1;
    off[i + 1] = off[i] + nrow[i];
    voff[i + 1] = voff[i] + d->gamma[i] + 1;
    doff[i + 1] = doff[i] + d->gamma[i];
    if (pre > 0) p.prefill = true;
  }
  p.M = off[p.B];
  p.Mv = voff[p.B];
  p.S = doff[p.B];
  p.Mp = (p.M + 31) / 32 * 32;
  if (forward) {
    p.d = m->d_model;
    p.nq = m->n_q_heads;
    p.nkv = m->n_kv_heads;
    p.hd = m->head_dim;
    p.F = m->d_ff;
    p.V = m->vocab;
    p.G = p.nq / p.nkv;
    p.qdim = p.nq * p.hd;
    p.kvdim = p.nkv * p.hd;
    p.qkvN = p.qdim + 2 * p.kvdim;
    p.bf16 = m->dtype == WISP_BF16;
    for (int i = 0; i < p.B; ++i) p.max_tokens = std::max(p.max_tokens, d->ctx_len[i] + nrow[i]);
    if (p.bf16) {
      p.g_qkv = gemm_bf16_plan(p.M, p.qkvN, p.d);
      p.g_o = gemm_bf16_plan(p.M, p.d, p.qdim);
      p.g_gu = gemm_bf16_plan(p.M, 2 * p.F, p.d);
      p.g_down = gemm_bf16_plan(p.M, p.d, p.F);
      p.g_lm = gemm_bf16_plan(p.Mv, p.V, p.d);
      p.g_lm.splits = 1;
      p.g_lm.kf_per_split = p.d / 16;
      // split-KV work list: items of <= 48 query rows and a run of page pairs.  One wave per
      // item and one 4-wave workgroup per CU are resident at a time, so a round started by
      // a few left-over workgroups would double the kernel's time; an item spans at most
      // kAttnMaxChunkPages pages, whose block ids one wave keeps in a register.
      const int64_t slots = 4 * (int64_t)device_cus();
      // items of a group: its page pairs split into n equal parts (n = ceil(pairs / L)),
      // L being the shortest item length (in pairs) whose items fill whole rounds of the
      // device's wave slots; equal parts keep every wave's item close to L pairs, so no
      // wave waits on a longer one
      // a row group's keys end at its last row's causal limit (prompt rows see fewer)
      auto group_tokens = [&](int i, int g) {
        const int rows = nrow[i] * p.G;
        const int last = std::min(rows, (g + 1) * kAttnRowsPerItem) - 1;
        return d->ctx_len[i] + last / p.G + 1;
      };
      auto count_items = [&](int L) {
        int64_t n = 0;
        for (int i = 0; i < p.B; ++i) {
          const int nrbg = (nrow[i] * p.G + kAttnRowsPerItem - 1) / kAttnRowsPerItem;
          for (int g = 0; g < nrbg; ++g) {
            const int64_t pairs = (group_tokens(i, g) + 31) / 32;
            n += (int64_t)p.nkv * ((pairs + L - 1) / L);
          }
        }
        return n;
      };
      const int L_max = kAttnMaxChunkPages / 2;
      int64_t rounds = 1;
      const int64_t fewest = count_items(L_max);
      // the work list holds at most fewest + slots items (below); its indices are int
      if (fewest > kAttnMaxItems - slots)
        return fail(WISP_E_UNSUPPORTED, "the batch's contexts need %lld attention work items (at most %d)",
                    (long long)fewest, kAttnMaxItems - (int)slots);
      while (rounds * slots < fewest) ++rounds;
      int L = 2;
      while (L < L_max && count_items(L) > rounds * slots) ++L;
      // Small batches leave wave slots idle even at the shortest items, and their step is
      // latency-bound: longer items then cost little, while a group of more than
      // kAttnCombineChunks chunks costs the combine further dependent loads.  Whenever the
      // items still fit one round of the wave slots, they grow until no group has more
      // than kAttnCombineChunks of them (B = 1: attention + combine 10.4 + 13.9 -> 14.3 +
      // 4.2 us per layer; B = 16: 27.7 -> 25.5 us; B = 4 and 8 within 3 %).
      {
        int64_t most = 0;
        for (int i = 0; i < p.B; ++i) {
          const int nrbg = (nrow[i] * p.G + kAttnRowsPerItem - 1) / kAttnRowsPerItem;
          for (int g = 0; g < nrbg; ++g) most = std::max<int64_t>(most, (group_tokens(i, g) + 31) / 32);
        }
        const int Lc = (int)std::min<int64_t>(L_max, std::max<int64_t>(L, (most + kAttnCombineChunks - 1) / kAttnCombineChunks));
        if (count_items(Lc) <= slots) L = Lc;
      }
      for (int i = 0; i < p.B; ++i) {
        const int rows = nrow[i] * p.G;
        const int nrbg = (rows + kAttnRowsPerItem - 1) / kAttnRowsPerItem;
        for (int h = 0; h < p.nkv; ++h)
          for (int g = 0; g < nrbg; ++g) {
            const int T = group_tokens(i, g);
            const int pairs = (T + 31) / 32;
            const int n = (pairs + L - 1) / L;
            AttnGroup gr{};
            gr.req = i;
            gr.kvh = h;
            gr.rbg = g;
            gr.first_item = (int32_t)p.items.size();
            for (int k = 0; k < n; ++k) {
              AttnItem it{};
              it.req = i;
              it.kvh_rbg = h | (g << 16);
              it.t0 = 32 * (int)((int64_t)k * pairs / n);
              it.t1 = std::min(T, 32 * (int)((int64_t)(k + 1) * pairs / n));
              p.items.push_back(it);
            }
            gr.n_items = (int32_t)p.items.size() - gr.first_item;
            p.max_group_chunks = std::max(p.max_group_chunks, (int)gr.n_items);
            p.groups.push_back(gr);
          }
      }
    }
  }
  // descriptor block
  size_t n = 0;
  auto take = [&](size_t &f, size_t cnt) {
    f = n;
    n += (cnt + 63) / 64 * 64;
  };
  take(p.i_off, p.B + 1);
  take(p.i_doff, p.B + 1);
  take(p.i_gamma, p.B);
  take(p.i_ctx, p.B);
  take(p.i_req, p.B);
  take(p.i_row_req, p.M);
  take(p.i_row_pos, p.M);
  take(p.i_items, p.items.size() * 4);
  take(p.i_groups, p.groups.size() * 8);
  take(p.i_voff, p.B + 1);
  take(p.i_nrow, p.B);
  take(p.i_vrow, p.Mv);
  p.host.assign(n, 0);
  for (int i = 0; i <= p.B; ++i) {
    p.host[p.i_off + i] = off[i];
    p.host[p.i_doff + i] = doff[i];
    p.host[p.i_voff + i] = voff[i];
  }
  for (int i = 0; i < p.B; ++i) {
    p.host[p.i_gamma + i] = d->gamma[i];
    p.host[p.i_ctx + i] = d->ctx_len[i];
    p.host[p.i_req + i] = d->req_id ? (int32_t)d->req_id[i] : i;
    p.host[p.i_nrow + i] = nrow[i];
    for (int j = 0; j < nrow[i]; ++j) {
      p.host[p.i_row_req + off[i] + j] = i;
      p.host[p.i_row_pos + off[i] + j] = d->ctx_len[i] + j;
    }
    for (int j = 0; j <= d->gamma[i]; ++j) p.host[p.i_vrow + voff[i] + j] = off[i + 1] - (d->gamma[i] + 1) + j;
  }
  if (!p.items.empty()) std::memcpy(&p.host[p.i_items], p.items.data(), p.items.size() * sizeof(AttnItem));
  if (!p.groups.empty()) std::memcpy(&p.host[p.i_groups], p.groups.data(), p.groups.size() * sizeof(AttnGroup));

  // workspace
  size_t w = 0;
  carve(w, p.w_err, 256);
  carve(w, p.w_desc, p.host.size() * sizeof(int32_t));
  const int CH = sampler_chunks(std::max(p.V, 1));
  carve(w, p.w_sm, (size_t)p.Mv * CH * 4);
  carve(w, p.w_si, (size_t)p.Mv * CH * 4);
  carve(w, p.w_ss, (size_t)p.Mv * CH * 8);
  carve(w, p.w_vtok, (size_t)(p.prefill ? p.Mv : 0) * 4);
  carve(w, p.w_rk, (size_t)p.B * CH * 2 * 4);
  carve(w, p.w_ri, (size_t)p.B * CH * 2 * 4);
  carve(w, p.w_rR, (size_t)p.B * 4);
  if (forward) {
    const size_t es = p.bf16 ? 2 : 4;
    carve(w, p.w_rope, (size_t)p.M * p.hd * 4);
    carve(w, p.w_h, (size_t)p.M * p.d * 4);
    carve(w, p.w_xn, (size_t)p.Mp * p.d * es);
    carve(w, p.w_ao, (size_t)p.Mp * p.qdim * es);
    carve(w, p.w_af, (size_t)p.Mp * p.F * es);
    carve(w, p.w_q, (size_t)p.M * p.qdim * es);
    size_t part = 0;
    if (p.bf16) {
      part = std::max({(size_t)p.g_qkv.splits * p.qkvN, (size_t)p.g_o.splits * p.d,
                       (size_t)p.g_gu.splits * 2 * p.F, (size_t)p.g_down.splits * p.d});
    } else {
      part = std::max({(size_t)p.qkvN, (size_t)p.d, (size_t)2 * p.F});
    }
    carve(w, p.w_part, part * p.M * 4);
    carve(w, p.w_attn_o, p.items.size() * (size_t)p.hd * 64 * 4);
    carve(w, p.w_attn_ml, p.items.size() * 64 * 2 * 4);
    if (p.bf16) {
      p.lm_tiles = (p.V + p.g_lm.bn - 1) / p.g_lm.bn;
      carve(w, p.w_lmm, (size_t)p.Mv * p.lm_tiles * 4);
      carve(w, p.w_lmi, (size_t)p.Mv * p.lm_tiles * 4);
    }
  }
  p.total = w;
  return WISP_OK;
}

// ------------------------------------------------------------------------------------------
// optional per-kernel-class timing: while a class scope is open, every launch in it gets a
// pair of HIP events stamped with that dispatch's own begin and end (launch_timing_events);
// a class's time is the sum of its dispatches' durations, its launch count the number of
// scopes, and its bytes / flops are those of the scope
// ------------------------------------------------------------------------------------------
struct ProfRec {
  int kind;
  int scopes;                 // 1 on a scope's first dispatch, else 0
  double bytes, flops;        // the scope's figures, on its first dispatch
  hipEvent_t a, b;
};
struct ProfState {
  bool on = false;
  int open_kind = -1;         // class of the open scope (-1: none)
  bool open_first = false;    // no dispatch of the open scope recorded yet
  double open_bytes = 0, open_flops = 0;
  std::vector<ProfRec> pending;
  std::vector<hipEvent_t> free_events;
  double ms[WISP_PROF_KINDS] = {}, bytes[WISP_PROF_KINDS] = {}, flops[WISP_PROF_KINDS] = {};
  int64_t launches[WISP_PROF_KINDS] = {};
};
ProfState g_prof;

hipEvent_t prof_event() {
  if (!g_prof.free_events.empty()) {
    hipEvent_t e = g_prof.free_events.back();
    g_prof.free_events.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  (void)hipEventCreate(&e);
  return e;
}

struct ProfScope {   // opens a timing scope of class `kind` over the launches it encloses
  ProfScope(int kind, double bytes, double flops, hipStream_t) {
    if (g_prof.on) {
      g_prof.open_kind = kind;
      g_prof.open_first = true;
      g_prof.open_bytes = bytes;
      g_prof.open_flops = flops;
    }
  }
  ~ProfScope() { g_prof.open_kind = -1; }
};

void prof_collect() {
  for (auto &r : g_prof.pending) {
    (void)hipEventSynchronize(r.b);
    float ms = 0.f;
    (void)hipEventElapsedTime(&ms, r.a, r.b);
    g_prof.ms[r.kind] += ms;
    g_prof.bytes[r.kind] += r.bytes;
    g_prof.flops[r.kind] += r.flops;
    g_prof.launches[r.kind] += r.scopes;
    g_prof.free_events.push_back(r.a);
    g_prof.free_events.push_back(r.b);
  }
  g_prof.pending.clear();
}

}  // namespace

bool wisp::launch_timing_events(hipEvent_t *start, hipEvent_t *stop) {
  if (!g_prof.on || g_prof.open_kind < 0) return false;
  ProfRec r{g_prof.open_kind, 0, 0.0, 0.0, prof_event(), prof_event()};
  if (g_prof.open_first) {
    r.scopes = 1;
    r.bytes = g_prof.open_bytes;
    r.flops = g_prof.open_flops;
    g_prof.open_first = false;
  }
  g_prof.pending.push_back(r);
  *start = r.a;
  *stop = r.b;
  return true;
}

namespace {

// pinned staging for the descriptor upload, reused once the previous copy has finished
struct Staging {
  void *buf = nullptr;
  size_t cap = 0;
  hipEvent_t ev = nullptr;
  bool pending = false;
};
thread_local Staging g_stage;

wisp_status upload(const Plan &p, char *ws, hipStream_t s) {
  const size_t bytes = p.host.size() * sizeof(int32_t);
  if (bytes == 0) return WISP_OK;
  if (g_stage.pending) {
    if (hipEventSynchronize(g_stage.ev) != hipSuccess) return fail(WISP_E_HIP, "staging event sync failed");
    g_stage.pending = false;
  }
  if (g_stage.cap < bytes) {
    if (g_stage.buf) (void)hipHostFree(g_stage.buf);
    g_stage.buf = nullptr;
    g_stage.cap = 0;
    size_t cap = std::max<size_t>(bytes, 1 << 16);
    if (hipHostMalloc(&g_stage.buf, cap, hipHostMallocDefault) != hipSuccess)
      return fail(WISP_E_HIP, "pinned staging allocation failed");
    g_stage.cap = cap;
  }
  if (!g_stage.ev && hipEventCreateWithFlags(&g_stage.ev, hipEventDisableTiming) != hipSuccess)
    return fail(WISP_E_HIP, "event creation failed");
  std::memcpy(g_stage.buf, p.host.data(), bytes);
  if (hipMemcpyAsync(ws + p.w_desc, g_stage.buf, bytes, hipMemcpyHostToDevice, s) != hipSuccess)
    return fail(WISP_E_HIP, "descriptor upload failed");
  if (hipEventRecord(g_stage.ev, s) != hipSuccess) return fail(WISP_E_HIP, "event record failed");
  g_stage.pending = true;
  return WISP_OK;
}

SamplerScratch sampler_scratch(const Plan &p, char *ws) {
  SamplerScratch sc;
  sc.part_m = reinterpret_cast<float *>(ws + p.w_sm);
  sc.part_i = reinterpret_cast<int32_t *>(ws + p.w_si);
  sc.part_s = reinterpret_cast<double *>(ws + p.w_ss);
  sc.race_k = reinterpret_cast<float *>(ws + p.w_rk);
  sc.race_i = reinterpret_cast<int32_t *>(ws + p.w_ri);
  sc.req_R = reinterpret_cast<int32_t *>(ws + p.w_rR);
  return sc;
}

StepDesc step_desc(const Plan &p, char *ws, const wisp_batch_desc *d, int n_blocks, int *err = nullptr) {
  const int32_t *base = reinterpret_cast<const int32_t *>(ws + p.w_desc);
  StepDesc sd;
  sd.off = base + p.i_off;
  sd.doff = base + p.i_doff;
  sd.gamma = base + p.i_gamma;
  sd.ctx = base + p.i_ctx;
  sd.req_id = reinterpret_cast<const uint32_t *>(base + p.i_req);
  sd.row_req = base + p.i_row_req;
  sd.row_pos = base + p.i_row_pos;
  sd.nrow = base + p.i_nrow;
  sd.page_table = d->kv_page_table;
  sd.pt_stride = d->pt_stride;
  sd.n_blocks = n_blocks;
  sd.err = err ? err : reinterpret_cast<int *>(ws + p.w_err);
  return sd;
}

// the LM head's per-tile row maxima (bf16 path), which spare the sampler a pass over the logits
RowMaxOut lm_row_max(const Plan &p, char *ws) {
  if (!p.bf16 || p.lm_tiles == 0) return RowMaxOut{nullptr, nullptr, 0};
  return RowMaxOut{reinterpret_cast<float *>(ws + p.w_lmm), reinterpret_cast<int32_t *>(ws + p.w_lmi), p.lm_tiles};
}

int gemm_class(const Plan &p, const GemmCfg &c) {
  if (!p.bf16) return WISP_PROF_GEMM_TILED;
  if (c.kind == 4) return WISP_PROF_GEMM_TILE;
  return c.kind == 2 ? WISP_PROF_GEMM_RING2 : WISP_PROF_GEMM_RING1;
}

wisp_status hip_check(const char *what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(WISP_E_HIP, "%s: %s", what, hipGetErrorString(e));
  return WISP_OK;
}

template <typename T>
wisp_status run_forward(const Plan &p, const wisp_model *m, const wisp_kv *kv, const StepDesc &sd,
                        char *ws, const int32_t *tokens, float *logits, hipStream_t s) {
  const bool packed = p.bf16;
  float *cs = reinterpret_cast<float *>(ws + p.w_rope);
  float *h = reinterpret_cast<float *>(ws + p.w_h);
  T *xn = reinterpret_cast<T *>(ws + p.w_xn);
  T *ao = reinterpret_cast<T *>(ws + p.w_ao);
  T *af = reinterpret_cast<T *>(ws + p.w_af);
  T *qb = reinterpret_cast<T *>(ws + p.w_q);
  float *part = reinterpret_cast<float *>(ws + p.w_part);
  const int64_t layer_elems = (int64_t)kv->n_blocks * p.nkv * WISP_PAGE * p.hd;
  const AttnItem *items = reinterpret_cast<const AttnItem *>(ws + p.w_desc + p.i_items * 4);
  const AttnGroup *groups = reinterpret_cast<const AttnGroup *>(ws + p.w_desc + p.i_groups * 4);
  const int32_t *vrow = reinterpret_cast<const int32_t *>(ws + p.w_desc) + p.i_vrow;

  const double es = p.bf16 ? 2.0 : 4.0;
  // algorithmic bytes of a projection: its weights, read once per step (activations and
  // results are a few percent at the step's row counts and not counted)
  auto gemm_bytes = [&](int N, int K) { return es * (double)N * K; };
  auto gemm_flops = [&](int N, int K) { return 2.0 * p.M * N * K; };
  const double kv_tok = 2.0 * p.nkv * p.hd * es;   // K and V bytes per token per layer
  double attn_bytes = 0.0, attn_flops = 0.0;
  for (const AttnItem &it : p.items) {
    const int G = p.G;
    const int rows = (int)p.host[p.i_nrow + it.req];
    const int rbg = it.kvh_rbg >> 16;
    const int nr = std::min(kAttnRowsPerItem, rows * G - rbg * kAttnRowsPerItem);
    if (rbg == 0) attn_bytes += (double)(it.t1 - it.t0) * kv_tok / p.nkv;
    attn_flops += 4.0 * p.hd * nr * (it.t1 - it.t0);
  }
  {
    ProfScope ps(WISP_PROF_ROWS, 0, 0, s);
    rope_table(sd, cs, p.M, p.hd, m->rope_base, s);
    embed_norm<T>(sd, (const T *)m->embed, (const T *)m->attn_norm[0], tokens, h, xn, packed, p.M, p.d,
                  p.V, m->rms_eps, s);
  }
  for (int l = 0; l < m->n_layers; ++l) {
    T *kl = (T *)kv->k_pool + l * layer_elems;
    T *vl = (T *)kv->v_pool + l * layer_elems;
    // one dense projection: C = act . W^T (fp32 partials over cfg.splits K ranges)
    auto gemm = [&](const T *act, const void *w, float *out, int N, int K, const GemmCfg &cfg) {
      ProfScope ps(gemm_class(p, cfg), gemm_bytes(N, K), gemm_flops(N, K), s);
      if (p.bf16)
        gemm_bf16((const uint16_t *)act, (const uint16_t *)w, out, p.M, N, K, N, cfg, s);
      else
        gemm_f32((const float *)act, (const float *)w, out, p.M, N, K, N, s);
      return p.bf16 ? cfg.splits : 1;
    };
    const int sq = gemm(xn, m->w_qkv[l], part, p.qkvN, p.d, p.g_qkv);
    {
      ProfScope ps(WISP_PROF_ROWS, 0, 0, s);
      qkv_rope_append<T>(sd, part, sq, cs, qb, kl, vl, p.M, p.nq, p.nkv, p.hd, s);
    }
    if (p.bf16) {
      float *po = reinterpret_cast<float *>(ws + p.w_attn_o);
      float *pml = reinterpret_cast<float *>(ws + p.w_attn_ml);
      {
        ProfScope ps(WISP_PROF_ATTN, attn_bytes, attn_flops, s);
        attention_bf16_main(sd, items, (int)p.items.size(), (const uint16_t *)qb, (const uint16_t *)kl,
                            (const uint16_t *)vl, po, pml, p.nq, p.nkv, p.hd, s);
      }
      ProfScope ps(WISP_PROF_ATTN_COMBINE, 0, 0, s);
      attention_bf16_combine(sd, groups, (int)p.groups.size(), p.max_group_chunks, po, pml, (uint16_t *)ao, true, p.qdim, p.nq,
                             p.nkv, p.hd, s);
    } else {
      ProfScope ps(WISP_PROF_ATTN, attn_bytes, attn_flops, s);
      attention_f32(sd, p.B, (const float *)qb, (const float *)kl, (const float *)vl, (float *)ao, p.nq,
                    p.nkv, p.hd, p.max_tokens, s);
    }
    const int so = gemm(ao, m->w_o[l], part, p.d, p.qdim, p.g_o);
    {
      ProfScope ps(WISP_PROF_ROWS, 0, 0, s);
      resid_norm<T>(part, so, h, (const T *)m->mlp_norm[l], xn, packed, p.M, p.d, m->rms_eps, s);
    }
    if (p.bf16 && p.g_gu.kind == 4 && p.g_gu.splits == 1) {
      // one K range on the tile kernel: SwiGLU in the GEMM's epilogue, which writes the down
      // projection's bf16 input directly (no fp32 gate/up round trip, no SwiGLU launch)
      ProfScope ps(gemm_class(p, p.g_gu), gemm_bytes(2 * p.F, p.d), gemm_flops(2 * p.F, p.d), s);
      gemm_bf16((const uint16_t *)xn, (const uint16_t *)m->w_gate_up[l], part, p.M, 2 * p.F, p.d, 2 * p.F, p.g_gu,
                s, RowMaxOut{nullptr, nullptr, 0}, SwigluOut{(uint16_t *)af, p.F});
    } else {
      const int sg = gemm(xn, m->w_gate_up[l], part, 2 * p.F, p.d, p.g_gu);
      ProfScope ps(WISP_PROF_ROWS, 0, 0, s);
      swiglu<T>(part, sg, af, packed, p.M, p.F, p.bf16, s);   // bf16 gate/up: interleaved columns
    }
    const int sdn = gemm(af, m->w_down[l], part, p.d, p.F, p.g_down);
    const bool last = l + 1 == m->n_layers;
    const T *gain = last ? (const T *)m->final_norm : (const T *)m->attn_norm[l + 1];
    {
      ProfScope ps(WISP_PROF_ROWS, 0, 0, s);
      if (last && p.prefill)   // only the verification rows reach the LM head: compact them
        resid_norm<T>(part, sdn, h, gain, xn, packed, p.M, p.d, m->rms_eps, s, vrow, p.Mv);
      else
        resid_norm<T>(part, sdn, h, gain, xn, packed, p.M, p.d, m->rms_eps, s);
    }
  }
  {
    const double lm_bytes = es * (double)p.V * p.d;
    ProfScope ps(gemm_class(p, p.g_lm), lm_bytes, 2.0 * p.Mv * p.V * p.d, s);
    if (p.bf16)
      gemm_bf16((const uint16_t *)xn, (const uint16_t *)m->lm_head, logits, p.Mv, p.V, p.d, p.V, p.g_lm, s,
                lm_row_max(p, ws));
    else
      gemm_f32((const float *)xn, (const float *)m->lm_head, logits, p.Mv, p.V, p.d, p.V, s);
  }
  return hip_check("forward launch");
}

}  // namespace

namespace {

// validation shared by the two verification entry points
wisp_status check_verify(const wisp_model *model, const wisp_kv *kv, const wisp_batch_desc *desc,
                         const int32_t *tokens, const int32_t *accept_len, const int32_t *out_tokens) {
  wisp_status st;
  if ((st = check_model(model, true)) != WISP_OK) return st;
  if ((st = check_desc(desc, true, true)) != WISP_OK) return st;
  if (desc->B == 0) return WISP_OK;
  if (!kv || !kv->k_pool || !kv->v_pool) return fail(WISP_E_INVALID, "KV pools are NULL");
  if (kv->page_size != WISP_PAGE) return fail(WISP_E_UNSUPPORTED, "page_size must be %d", WISP_PAGE);
  if (kv->n_blocks <= 0) return fail(WISP_E_INVALID, "n_blocks must be positive");
  if (!tokens || !accept_len || !out_tokens) return fail(WISP_E_INVALID, "NULL tokens / outputs");
  return WISP_OK;
}

wisp_status plan_verify(Plan &p, const wisp_model *model, const wisp_batch_desc *desc, const float *draft_probs) {
  wisp_status st;
  if ((st = make_plan(p, model, desc, true)) != WISP_OK) return st;
  if (p.S > 0 && !draft_probs) return fail(WISP_E_INVALID, "draft_probs is NULL");
  if (!p.bf16 && p.max_tokens > 32768) return fail(WISP_E_UNSUPPORTED, "fp32 path supports <= 32768 tokens per request");
  return WISP_OK;
}

// the step's kernel sequence on a planned, uploaded workspace `ws`; `err` (or NULL: the
// workspace's own record) receives the device-side input faults
wisp_status run_verify(const Plan &p, const wisp_model *model, const wisp_kv *kv, const wisp_batch_desc *desc,
                       const int32_t *tokens, const float *draft_probs, uint64_t rng_seed, int32_t *accept_len,
                       int32_t *out_tokens, float *target_logits, char *ws, int *err, hipStream_t s) {
  wisp_status st;
  StepDesc sd = step_desc(p, ws, desc, kv->n_blocks, err);
  if (p.bf16)
    st = run_forward<uint16_t>(p, model, kv, sd, ws, tokens, target_logits, s);
  else
    st = run_forward<float>(p, model, kv, sd, ws, tokens, target_logits, s);
  if (st != WISP_OK) return st;
  // the acceptance sees the verification rows only: row offsets over them, and (with
  // prompt rows present) their tokens gathered into a compact array
  StepDesc sv = sd;
  sv.off = reinterpret_cast<const int32_t *>(ws + p.w_desc) + p.i_voff;
  const int32_t *vtok = tokens;
  if (p.prefill) {
    int32_t *g = reinterpret_cast<int32_t *>(ws + p.w_vtok);
    gather_ints(tokens, reinterpret_cast<const int32_t *>(ws + p.w_desc) + p.i_vrow, p.Mv, g, s);
    vtok = g;
  }
  // algorithmic bytes: one fp32 pass over the logits (the maxima come with the LM head in
  // bf16; the fp32 path makes two passes) plus one logits row and one q row per request
  const RowMaxOut lm = lm_row_max(p, ws);
  ProfScope ps(WISP_PROF_SAMPLER, (lm.m ? 1.0 : 2.0) * p.Mv * p.V * 4.0 + 2.0 * p.B * p.V * 4.0, 0, s);
  sampler(sv, p.B, p.Mv, p.V, target_logits, vtok, draft_probs, desc->temperature, rng_seed,
          sampler_scratch(p, ws), accept_len, out_tokens, s, lm);
  return hip_check("sampler launch");
}

}  // namespace

// ------------------------------------------------------------------------------------------
// Scratch of the allocation-free entry point: one static array, of which every GPU the
// library runs on holds its own copy (at its own address, looked up once per device).
// Host code never uses the array's name as an address, only the looked-up pointer.
// ------------------------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[WISP_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

wisp_status noalloc_scratch(char **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return fail(WISP_E_HIP, "hipGetDevice failed");
  if (dev < 0 || dev >= kMaxDevices) return fail(WISP_E_UNSUPPORTED, "device %d", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(WISP_E_HIP, "scratch address on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = static_cast<char *>(g_scratch_ptr[dev]);
  return WISP_OK;
}

// The descriptor block reaches the device as kernel arguments, a few KB per launch: no
// pinned staging buffer and no host copy that must outlive the call.
constexpr int kDescChunkInts = 960;
struct DescChunk {
  int32_t n;
  int32_t v[kDescChunkInts];
};

__global__ void put_desc_kernel(DescChunk c, int32_t *__restrict__ dst) {
  for (int i = threadIdx.x; i < c.n; i += blockDim.x) dst[i] = c.v[i];
}

wisp_status upload_by_arguments(const Plan &p, char *ws, hipStream_t s) {
  int32_t *dst = reinterpret_cast<int32_t *>(ws + p.w_desc);
  const size_t n = p.host.size();
  DescChunk c;
  for (size_t o = 0; o < n; o += kDescChunkInts) {
    c.n = (int32_t)std::min<size_t>(kDescChunkInts, n - o);
    std::memcpy(c.v, p.host.data() + o, (size_t)c.n * sizeof(int32_t));
    launch(put_desc_kernel, 1, 256, 0, s, c, dst + o);
  }
  return hip_check("descriptor upload");
}

}  // namespace

namespace wisp {
// lets the host-only sources (the scheduler, the KV manager) report through wisp_last_error
wisp_status report_error(wisp_status st, const char *msg) { return fail(st, "%s", msg); }
wisp_status report_exception(const char *who, bool out_of_memory) {
  return out_of_memory ? fail(WISP_E_HOST_MEMORY, "%s: host memory exhausted", who)
                       : fail(WISP_E_INVALID, "%s: unexpected host-side exception", who);
}
}  // namespace wisp

// ------------------------------------------------------------------------------------------
// exported entry points
// ------------------------------------------------------------------------------------------
extern "C" {

const char *wisp_last_error(void) { return g_last_error; }

size_t wisp_workspace_size(const wisp_model *model, const wisp_batch_desc *desc) {
  return guarded_size([&]() -> size_t {
    if (check_model(model, false) != WISP_OK || check_desc(desc, false, true) != WISP_OK) return 0;
    Plan p;
    if (make_plan(p, model, desc, true) != WISP_OK) return 0;
    return p.total;
  });
}

size_t wisp_logits_workspace_size(const wisp_model *model, const wisp_batch_desc *desc) {
  return guarded_size([&]() -> size_t {
    if (check_model(model, false) != WISP_OK || check_desc(desc, false, true) != WISP_OK) return 0;
    Plan p;
    if (make_plan(p, model, desc, true) != WISP_OK) return 0;
    return align256((size_t)p.Mv * (size_t)p.V * sizeof(float));
  });
}

size_t wisp_accept_workspace_size(const wisp_batch_desc *desc, int32_t vocab) {
  return guarded_size([&]() -> size_t {
    if (check_desc(desc, false, false) != WISP_OK || vocab <= 0) return 0;
    Plan p;
    if (make_plan(p, nullptr, desc, false, vocab) != WISP_OK) return 0;
    return p.total;
  });
}

wisp_status wisp_pack_gate_up(void *dst, const void *w_gate, const void *w_up, int32_t d_ff, int32_t d_model,
                              int32_t dtype, void *stream) {
  return guarded("wisp_pack_gate_up", [&]() -> wisp_status {
    if (!dst || !w_gate || !w_up) return fail(WISP_E_INVALID, "NULL pointer");
    if (d_ff <= 0 || d_model <= 0) return fail(WISP_E_INVALID, "d_ff, d_model must be positive");
    hipStream_t s = (hipStream_t)stream;
    if (dtype == WISP_BF16) {
      if (d_ff % 32 || d_model % 16)
        return fail(WISP_E_UNSUPPORTED, "bf16 packing needs d_ff %% 32 == 0 and d_model %% 16 == 0");
      pack_gate_up_bf16((uint16_t *)dst, (const uint16_t *)w_gate, (const uint16_t *)w_up, d_ff, d_model, s);
    } else if (dtype == WISP_F32) {
      const size_t half = (size_t)d_ff * d_model * 4;
      if (hipMemcpyAsync(dst, w_gate, half, hipMemcpyDeviceToDevice, s) != hipSuccess ||
          hipMemcpyAsync((char *)dst + half, w_up, half, hipMemcpyDeviceToDevice, s) != hipSuccess)
        return fail(WISP_E_HIP, "copy failed");
    } else {
      return fail(WISP_E_UNSUPPORTED, "dtype %d", dtype);
    }
    return hip_check("pack");
  });
}

wisp_status wisp_pack_linear(void *dst, const void *src, int32_t rows, int32_t cols, int32_t dtype,
                             void *stream) {
  return guarded("wisp_pack_linear", [&]() -> wisp_status {
    if (!dst || !src) return fail(WISP_E_INVALID, "NULL pointer");
    if (rows <= 0 || cols <= 0) return fail(WISP_E_INVALID, "rows, cols must be positive");
    hipStream_t s = (hipStream_t)stream;
    if (dtype == WISP_BF16) {
      if (rows % 32 || cols % 16) return fail(WISP_E_UNSUPPORTED, "bf16 packing needs rows %% 32 == 0 and cols %% 16 == 0");
      pack_linear_bf16((uint16_t *)dst, (const uint16_t *)src, rows, cols, s);
    } else if (dtype == WISP_F32) {
      if (hipMemcpyAsync(dst, src, (size_t)rows * cols * 4, hipMemcpyDeviceToDevice, s) != hipSuccess)
        return fail(WISP_E_HIP, "copy failed");
    } else {
      return fail(WISP_E_UNSUPPORTED, "dtype %d", dtype);
    }
    return hip_check("pack");
  });
}

wisp_status wisp_verify(const wisp_model *model, const wisp_kv *kv, const wisp_batch_desc *desc,
                        const int32_t *tokens, const float *draft_probs, uint64_t rng_seed,
                        int32_t *accept_len, int32_t *out_tokens, float *target_logits,
                        void *workspace, size_t workspace_bytes, void *stream) {
  return guarded("wisp_verify", [&]() -> wisp_status {
    wisp_status st;
    if ((st = check_verify(model, kv, desc, tokens, accept_len, out_tokens)) != WISP_OK) return st;
    if (desc->B == 0) return WISP_OK;
    if (!workspace) return fail(WISP_E_INVALID, "NULL workspace");
    Plan p;
    if ((st = plan_verify(p, model, desc, draft_probs)) != WISP_OK) return st;
    // without a caller buffer the logits live in the workspace, after everything else
    const size_t need = p.total + (target_logits ? 0 : align256((size_t)p.Mv * (size_t)p.V * sizeof(float)));
    if (workspace_bytes < need)
      return fail(WISP_E_WORKSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, need);
    hipStream_t s = (hipStream_t)stream;
    char *ws = (char *)workspace;
    if (!target_logits) target_logits = reinterpret_cast<float *>(ws + p.total);
    if ((st = upload(p, ws, s)) != WISP_OK) return st;
    return run_verify(p, model, kv, desc, tokens, draft_probs, rng_seed, accept_len, out_tokens, target_logits,
                      ws, nullptr, s);
  });
}

wisp_status wisp_verify_noalloc(const wisp_model *model, const wisp_kv *kv, const wisp_batch_desc *desc,
                                const int32_t *tokens, const float *draft_probs, uint64_t rng_seed,
                                int32_t *accept_len, int32_t *out_tokens, float *target_logits, int32_t *fault,
                                void *stream) {
  return guarded("wisp_verify_noalloc", [&]() -> wisp_status {
    wisp_status st;
    if ((st = check_verify(model, kv, desc, tokens, accept_len, out_tokens)) != WISP_OK) return st;
    if (desc->B == 0) return WISP_OK;
    Plan p;
    if ((st = plan_verify(p, model, desc, draft_probs)) != WISP_OK) return st;
    const size_t need = p.total + (target_logits ? 0 : align256((size_t)p.Mv * (size_t)p.V * sizeof(float)));
    if (need > (size_t)WISP_NOALLOC_SCRATCH_BYTES)
      return fail(WISP_E_WORKSPACE, "the batch needs %zu bytes of scratch, more than the %zu of the static "
                  "per-device scratch (use wisp_verify with a workspace)", need, (size_t)WISP_NOALLOC_SCRATCH_BYTES);
    char *ws = nullptr;
    if ((st = noalloc_scratch(&ws)) != WISP_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    if (!target_logits) target_logits = reinterpret_cast<float *>(ws + p.total);
    if ((st = upload_by_arguments(p, ws, s)) != WISP_OK) return st;
    return run_verify(p, model, kv, desc, tokens, draft_probs, rng_seed, accept_len, out_tokens, target_logits,
                      ws, fault, s);
  });
}

wisp_status wisp_accept(const wisp_batch_desc *desc, int32_t vocab, const float *logits,
                        const int32_t *tokens, const float *draft_probs, uint64_t rng_seed,
                        int32_t *accept_len, int32_t *out_tokens, void *workspace,
                        size_t workspace_bytes, void *stream) {
  return guarded("wisp_accept", [&]() -> wisp_status {
    wisp_status st;
    if ((st = check_desc(desc, false, false)) != WISP_OK) return st;
    if (desc->B == 0) return WISP_OK;
    if (vocab <= 0) return fail(WISP_E_INVALID, "vocab must be positive");
    if (!logits || !tokens || !accept_len || !out_tokens || !workspace)
      return fail(WISP_E_INVALID, "NULL logits / tokens / outputs / workspace");
    Plan p;
    if ((st = make_plan(p, nullptr, desc, false, vocab)) != WISP_OK) return st;
    if (p.S > 0 && !draft_probs) return fail(WISP_E_INVALID, "draft_probs is NULL");
    if (workspace_bytes < p.total)
      return fail(WISP_E_WORKSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, p.total);
    hipStream_t s = (hipStream_t)stream;
    char *ws = (char *)workspace;
    if ((st = upload(p, ws, s)) != WISP_OK) return st;
    StepDesc sd = step_desc(p, ws, desc, 0);
    sampler(sd, p.B, p.M, vocab, logits, tokens, draft_probs, desc->temperature, rng_seed,
            sampler_scratch(p, ws), accept_len, out_tokens, s);
    return hip_check("sampler launch");
  });
}

wisp_status wisp_attention(const wisp_model *model, const wisp_kv *kv, const wisp_batch_desc *desc,
                           const void *q, void *out, void *workspace, size_t workspace_bytes,
                           void *stream) {
  return guarded("wisp_attention", [&]() -> wisp_status {
    wisp_status st;
    if ((st = check_model(model, false)) != WISP_OK) return st;
    if ((st = check_desc(desc, true, true)) != WISP_OK) return st;
    if (desc->B == 0) return WISP_OK;
    if (!kv || !kv->k_pool || !kv->v_pool || kv->n_blocks <= 0) return fail(WISP_E_INVALID, "KV pools");
    if (kv->page_size != WISP_PAGE) return fail(WISP_E_UNSUPPORTED, "page_size must be %d", WISP_PAGE);
    if (!q || !out || !workspace) return fail(WISP_E_INVALID, "NULL q / out / workspace");
    Plan p;
    if ((st = make_plan(p, model, desc, true)) != WISP_OK) return st;
    if (!p.bf16 && p.max_tokens > 32768) return fail(WISP_E_UNSUPPORTED, "fp32 path supports <= 32768 tokens per request");
    if (workspace_bytes < p.total)
      return fail(WISP_E_WORKSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, p.total);
    hipStream_t s = (hipStream_t)stream;
    char *ws = (char *)workspace;
    if ((st = upload(p, ws, s)) != WISP_OK) return st;
    StepDesc sd = step_desc(p, ws, desc, kv->n_blocks);
    if (p.bf16) {
      const AttnItem *items = reinterpret_cast<const AttnItem *>(ws + p.w_desc + p.i_items * 4);
      const AttnGroup *groups = reinterpret_cast<const AttnGroup *>(ws + p.w_desc + p.i_groups * 4);
      float *po = reinterpret_cast<float *>(ws + p.w_attn_o);
      float *pml = reinterpret_cast<float *>(ws + p.w_attn_ml);
      attention_bf16_main(sd, items, (int)p.items.size(), (const uint16_t *)q, (const uint16_t *)kv->k_pool,
                          (const uint16_t *)kv->v_pool, po, pml, p.nq, p.nkv, p.hd, s);
      attention_bf16_combine(sd, groups, (int)p.groups.size(), p.max_group_chunks, po, pml, (uint16_t *)out, false, p.qdim, p.nq,
                             p.nkv, p.hd, s);
    } else {
      attention_f32(sd, p.B, (const float *)q, (const float *)kv->k_pool, (const float *)kv->v_pool,
                    (float *)out, p.nq, p.nkv, p.hd, p.max_tokens, s);
    }
    return hip_check("attention launch");
  });
}

wisp_status wisp_uniform(uint64_t rng_seed, uint32_t req_id, uint32_t tag, uint32_t row, uint32_t n,
                         float *out, void *stream) {
  return guarded("wisp_uniform", [&]() -> wisp_status {
    if (!out && n) return fail(WISP_E_INVALID, "out is NULL");
    uniform_draws(rng_seed, req_id, tag, row, n, out, (hipStream_t)stream);
    return hip_check("uniform launch");
  });
}

wisp_status wisp_profile_enable(int on) {
  return guarded("wisp_profile_enable", [&]() -> wisp_status {
    if (!on) prof_collect();
    g_prof.on = on != 0;
    return WISP_OK;
  });
}

wisp_status wisp_profile_read(int kind, double *ms, int64_t *launches, double *bytes, double *flops) {
  return guarded("wisp_profile_read", [&]() -> wisp_status {
    if (kind < 0 || kind >= WISP_PROF_KINDS) return fail(WISP_E_INVALID, "profile kind %d", kind);
    prof_collect();
    if (ms) *ms = g_prof.ms[kind];
    if (launches) *launches = g_prof.launches[kind];
    if (bytes) *bytes = g_prof.bytes[kind];
    if (flops) *flops = g_prof.flops[kind];
    return WISP_OK;
  });
}

wisp_status wisp_profile_reset(void) {
  return guarded("wisp_profile_reset", [&]() -> wisp_status {
    prof_collect();
    for (int k = 0; k < WISP_PROF_KINDS; ++k) {
      g_prof.ms[k] = g_prof.bytes[k] = g_prof.flops[k] = 0.0;
      g_prof.launches[k] = 0;
    }
    return WISP_OK;
  });
}

wisp_status wisp_gemm_plan(int32_t M, int32_t N, int32_t K, int32_t out[4]) {
  return guarded("wisp_gemm_plan", [&]() -> wisp_status {
    if (!out) return fail(WISP_E_INVALID, "out is NULL");
    if (M < 1 || N < 1 || K < 1 || N % 32 || K % 16)
      return fail(WISP_E_INVALID, "M, N, K must be positive, N a multiple of 32, K of 16");
    const GemmCfg c = gemm_bf16_plan(M, N, K);
    out[0] = c.kind;
    out[1] = c.rb;
    out[2] = c.mt;
    out[3] = c.splits;
    return WISP_OK;
  });
}

wisp_status wisp_check(void *workspace, void *stream) {
  return guarded("wisp_check", [&]() -> wisp_status {
    if (!workspace) return fail(WISP_E_INVALID, "workspace is NULL");
    hipStream_t s = (hipStream_t)stream;
    if (hipStreamSynchronize(s) != hipSuccess) return fail(WISP_E_HIP, "stream synchronize failed");
    int err = 0;
    if (hipMemcpy(&err, workspace, sizeof(int), hipMemcpyDeviceToHost) != hipSuccess)
      return fail(WISP_E_HIP, "error word read failed");
    if (err) {
      int zero = 0;
      (void)hipMemcpy(workspace, &zero, sizeof(int), hipMemcpyHostToDevice);
      return fail(WISP_E_DEVICE_INPUT, "device-side input check failed:%s%s",
                  (err & kErrToken) ? " token id out of range" : "",
                  (err & kErrBlock) ? " block id out of range" : "");
    }
    return WISP_OK;
  });
}

}  // extern "C"
