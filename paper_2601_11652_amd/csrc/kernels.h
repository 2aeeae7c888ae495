// Host-side launchers of the gfx950 kernels (one translation unit per kernel family).
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace wisp {

// ----- kernel launch ---------------------------------------------------------------------
// While per-launch timing is on, launch_timing_events hands out a pair of HIP events and the
// launch goes through hipExtLaunchKernelGGL, which stamps them with the dispatch's own begin
// and end (the gap between dispatches is not counted); otherwise it is a plain launch.
bool launch_timing_events(hipEvent_t *start, hipEvent_t *stop);

template <typename... Formals, typename... Actuals>
inline void launch(void (*kernel)(Formals...), dim3 grid, dim3 block, uint32_t shm, hipStream_t s,
                   Actuals... args) {
  hipEvent_t a = nullptr, b = nullptr;
  if (launch_timing_events(&a, &b))
    hipExtLaunchKernelGGL(kernel, grid, block, shm, s, a, b, 0u, args...);
  else
    kernel<<<grid, block, shm, s>>>(args...);
}

// ----- GEMMs: C[z][M][ldc] (fp32) = A[M][K] . W[N][K]^T over the z-th K range ----------
struct GemmCfg {
  int kind;         // 1: weight ring NT=1 R=8, 2: weight ring NT=2 R=4,
                    // 3: weight ring NT=1 R=8 with 8 waves (two per SIMD on half the rows each),
                    // 4: LDS-staged output tiles (gemm_bf16_tile, `variant`)
  int variant;      // kind 4: tile shape (see gemm_bf16_tile)
  int mt;           // 32-row fragments of A held by every workgroup
  int rb;           // row blocks (grid rows): rb * mt fragments cover ceil(M/32)
  int bm, bn;       // tile rows / cols
  int splits;       // K splits (partial sums in fp32, summed in fixed order later)
  int kf_per_split; // 16-wide K fragments per split
};
GemmCfg gemm_bf16_plan(int M, int N, int K);
void gemm_bf16(const uint16_t *A_packed, const uint16_t *W_packed, float *C, int M, int N, int K,
               int ldc, const GemmCfg &cfg, hipStream_t s, RowMaxOut rm = RowMaxOut{nullptr, nullptr, 0},
               SwigluOut sw = SwigluOut{nullptr, 0});
void gemm_f32(const float *A, const float *W, float *C, int M, int N, int K, int ldc, hipStream_t s);
// LDS-staged output tiles (both operands staged through LDS): variant 1 is 192 x 128,
// 4 is 192 x 256, 6 is 64 x 128, 7 is 128 x 128, 12 is 384 x 128, 13 is 256 x 128 and
// 17 is 256 x 256 (rows x columns, 8 waves), 5 is 32 x 256 (4 waves).  K is
// cut into chunks of 16 ks (ks = tile_k_steps(variant)); a work item sums kc_split chunks
// into its own fp32 partial C[z] (z = its K range), C[0] alone when kc_split covers K.
struct TileShape { int bm, bn, ks; };
TileShape tile_shape(int variant);
void gemm_bf16_tile(const uint16_t *A_packed, const uint16_t *W_packed, float *C, int M, int N, int K, int ldc,
                    int variant, int kc_split, RowMaxOut rm, hipStream_t s, SwigluOut sw = SwigluOut{nullptr, 0});
void pack_linear_bf16(uint16_t *dst, const uint16_t *src, int rows, int cols, hipStream_t s);
// gate/up weights ([F][d] each) packed with their 32-row blocks interleaved: packed row
// block 2b = gate rows 32b .. 32b + 31, 2b + 1 = the up rows of the same b
void pack_gate_up_bf16(uint16_t *dst, const uint16_t *gate, const uint16_t *up, int F, int d, hipStream_t s);

// ----- per-row layers --------------------------------------------------------------------
struct StepDesc {         // device arrays carved from the workspace
  const int32_t *off;     // [B+1] first row of request i
  const int32_t *doff;    // [B+1] first draft row of request i
  const int32_t *gamma;   // [B]
  const int32_t *ctx;     // [B]
  const uint32_t *req_id; // [B]
  const int32_t *row_req; // [M]
  const int32_t *row_pos; // [M]
  const int32_t *nrow;    // [B] rows forwarded per request (prompt tokens, root, drafts)
  const int32_t *page_table;
  int pt_stride;
  int n_blocks;
  int *err;
};

void rope_table(const StepDesc &d, float *cs, int M, int hd, float base, hipStream_t s);

template <typename T>
void embed_norm(const StepDesc &d, const T *embed, const T *gain, const int32_t *tokens, float *h,
                T *xn, bool packed, int M, int dm, int V, float eps, hipStream_t s);

// h += sum of the split partials, xn = RMSNorm(h) * gain; rows (optional) maps each of the
// n_out output rows to its source row (NULL: n_out = M, identity)
template <typename T>
void resid_norm(const float *part, int splits, float *h, const T *gain, T *xn, bool packed, int M,
                int dm, float eps, hipStream_t s, const int32_t *rows = nullptr, int n_out = -1);
// dst[i] = src[idx[i]], i < n
void gather_ints(const int32_t *src, const int32_t *idx, int n, int32_t *dst, hipStream_t s);

template <typename T>
void qkv_rope_append(const StepDesc &d, const float *part, int splits, const float *cs, T *q,
                     T *k_pool, T *v_pool, int M, int nq, int nkv, int hd, hipStream_t s);

template <typename T>
void swiglu(const float *part, int splits, T *out, bool packed, int M, int F, bool interleaved, hipStream_t s);

// ----- attention ---------------------------------------------------------------------------
struct AttnItem {   // one wave's work: request, kv head, row group, token range
  int32_t req, kvh_rbg, t0, t1;
};
struct AttnGroup {  // the chunks of one (request, kv head, row group), combined in order
  int32_t req, kvh, rbg, first_item, n_items, pad0, pad1, pad2;
};
constexpr int kAttnRowsPerItem = 48;   // query rows one wave carries (3 blocks of 16)
constexpr int kAttnMaxItems = 1 << 22;  // split-KV work items of one call (int indices, workspace)
constexpr int kAcceptRowsMax = 1 << 29; // rows of one acceptance-only call (int offsets)
constexpr int kAttnMaxChunkPages = 64; // pages of one item (one block id per lane)
constexpr int kAttnCombineChunks = 8;  // chunks the combine loads per round of dependent loads

// split-KV partials of every item, then their fixed-order combine into `out`
void attention_bf16_main(const StepDesc &d, const AttnItem *items, int n_items, const uint16_t *q,
                         const uint16_t *k_pool, const uint16_t *v_pool, float *part_o, float *part_ml,
                         int nq, int nkv, int hd, hipStream_t s);
void attention_bf16_combine(const StepDesc &d, const AttnGroup *groups, int n_groups, int max_group_chunks,
                            const float *part_o, const float *part_ml, uint16_t *out, bool out_packed,
                            int out_K, int nq, int nkv, int hd, hipStream_t s);
void attention_f32(const StepDesc &d, int B, const float *q, const float *k_pool,
                   const float *v_pool, float *out, int nq, int nkv, int hd, int max_tokens,
                   hipStream_t s);

// ----- acceptance ----------------------------------------------------------------------------
struct SamplerScratch {   // carved from the workspace; sizes from sampler_chunks(V)
  float *part_m;          // [M][CH] chunk maxima
  int32_t *part_i;        // [M][CH] chunk argmax (greedy)
  double *part_s;         // [M][CH] chunk sums of exponentials
  float *race_k;          // [B][CH][2] chunk race winners (p race, residual race)
  int32_t *race_i;        // [B][CH][2]
  int32_t *req_R;         // [B] first rejection
};
int sampler_chunks(int V);
// lm: the LM head's per-tile row maxima of these logits (RowMaxOut), or m == NULL
void sampler(const StepDesc &d, int B, int M, int V, const float *logits, const int32_t *tokens,
             const float *q, float T, uint64_t seed, SamplerScratch sc, int32_t *accept_len,
             int32_t *out_tokens, hipStream_t s, RowMaxOut lm = RowMaxOut{nullptr, nullptr, 0});
void uniform_draws(uint64_t seed, uint32_t req, uint32_t tag, uint32_t row, uint32_t n, float *out,
                   hipStream_t s);
void clear_ints(int *p, int n, hipStream_t s);

}  // namespace wisp
