// Host launchers of the gfx950 kernels (one translation unit per family).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace darts {

// ---- init (k_init.hip)
// Row mapping of a logical [n_out][n_in] tensor into its physical matrix:
// phys_row = (r / grp_outer) * stride_outer + ((r % grp_outer) / grp_inner) * stride_inner
//            + (r % grp_outer) % grp_inner + row_off
struct RowMap {
  int64_t grp_outer, stride_outer, grp_inner, stride_inner, row_off;
};
RowMap rowmap_plain(int64_t n_out, int64_t row_off);
hipError_t launch_init_weights(void* dst, bool bf16, int64_t n_out, int64_t n_in, int64_t fan_in,
                               uint32_t tensor_id, uint32_t layer, uint64_t seed, RowMap map,
                               hipStream_t st);
// Copy a caller's row-major logical [n_out][n_in] tensor (fp32 or bf16) into
// its physical rows under map.
hipError_t launch_copy_rows(void* dst, const void* src, bool bf16, int64_t n_out, int64_t n_in, RowMap map,
                            hipStream_t st);
hipError_t launch_rope_table(float2* table, int max_pos, int hd, double theta, hipStream_t st);
// streaming read (HBM read-rate reference): kStreamReadBlocks x 256 threads,
// one float per wavefront written to sink
constexpr int kStreamReadBlocks = 2048;
hipError_t launch_stream_read(const void* src, int64_t n16, float* sink, hipStream_t st);
hipError_t launch_fill_uniform(void* dst, uint64_t n, uint32_t tensor, uint64_t seed, bool bf16,
                               hipStream_t st);
hipError_t launch_fill_kv_pool(void* k, void* v, int64_t n_pages, int hkv, int hd, uint64_t seed,
                               bool bf16, hipStream_t st);
hipError_t launch_iota_perm(int32_t* stack, int64_t n, uint64_t perm_seed, bool permute,
                            hipStream_t st);

// ---- GEMM (k_gemm.hip): C[M,N] (op)= A[M,K] * W[N,K]^T
enum Epi { EPI_F32 = 0, EPI_BF16 = 1, EPI_ADD_F32 = 2, EPI_SWIGLU = 3 };
size_t gemm_workspace_bytes(int M, int N, int K);
// x += A . W^T and xn = bf16(RMSNorm(x)) (bf16 operands); *fused says whether
// xn was written (split-K plans) or the caller must normalise
// bf16 C = A . W^T in fp32 when the plan keeps K whole (*n_split = 1), else
// only the plan's split-K partial sums into ws (*n_split planes of M*N floats)
hipError_t launch_gemm_f32_or_partials(const void* A, int lda, const void* W, int ldw, float* C,
                                       int ldc, int M, int N, int K, void* ws, size_t ws_bytes,
                                       hipStream_t st, int* n_split);
hipError_t launch_gemm_add_norm(const void* A, int lda, const void* W, int ldw, float* x, int ldx,
                                int M, int N, int K, void* ws, size_t ws_bytes, float eps,
                                void* xn, hipStream_t st, bool* fused);
hipError_t launch_gemm(bool bf16, const void* A, int lda, const void* W, int ldw, void* C, int ldc,
                       int M, int N, int K, int epi, void* ws, size_t ws_bytes, hipStream_t st);

// ---- elementwise (k_elem.hip)
// embedding gather; with xn != NULL (bf16 models) also xn = bf16(RMSNorm(x))
hipError_t launch_embed_norm(const void* table, const int32_t* tokens, const int32_t* rows_traj,
                             int n_rows, int d, int vocab, float eps, float* x, void* xn,
                             hipStream_t st);
hipError_t launch_embed_v(const void* table, bool bf16, const int32_t* tokens,
                          const int32_t* rows_traj, int n_rows, int d, int vocab, float* x,
                          hipStream_t st);
hipError_t launch_rmsnorm(const float* x, int n_rows, int d, float eps, void* out, bool bf16,
                          hipStream_t st);
// pos(r) = pos_mod ? r % pos_mod + pos_base : pos_base
hipError_t launch_rope_append2(const float* qkv, int n_split, int64_t split_stride, int n_rows,
                               int hq, int hkv, int hd, const int32_t* row_pt, int pos_mod,
                               int pos_base, const int32_t* page_table, int pt_stride,
                               int64_t n_pages, const float2* rope, void* q_out, void* k_pool,
                               void* v_pool, bool bf16, hipStream_t st);
hipError_t launch_gather_rows(const float* src, const int32_t* rows, int n, int d, float* dst,
                              hipStream_t st);

// Grouped bf16 GEMM (mixture of experts): group e owns rows [g_off[e],
// g_off[e] + g_cnt[e]) of A and C and the weights W + e * w_stride ([N][K],
// row stride ldw).  mtiles lists the non-empty row tiles of tile_rows rows
// (grouped_plan), e << 16 | tile, *n_mtiles of them (device values).
// N % 128 == 0, K % 64 == 0.  packed_w: W is in the strip layout of
// launch_pack_strips (ldw = K; SwiGLU epilogue only).
constexpr int kGroupedTileRows = 128;      // largest row tile
constexpr int kGroupedTileRowsGU = 96;     // gate/up row tile of large decode batches
constexpr int kGroupedTileRowsMin = 64;    // smallest row tile (sizes the tile lists)
// Plan for n_pairs routed (row, expert) pairs over E experts: the row tile
// of the tile list and the kernel family.  64-row tiles while an expert gets
// few rows (decode batches: the weights are streamed and half-empty 128-row
// tiles would double the operand traffic), 96-row tiles for the gate/up
// projection from 48 rows per expert (so an expert's weights are not
// streamed twice), 128-row tiles for large batches (the prefill: more reuse
// of each weight tile).  wdirect: the gate/up weights go straight into MFMA
// registers (from 2 rows per expert up to the prefill), otherwise through
// the LDS tile ring.  nt_w: the weights are loaded non-temporal (gate/up in
// every decode batch; down while no expert needs a second row tile, whose
// second pass over the same weights would then miss the cache).
struct GroupedPlan {
  int tile_rows;
  bool wdirect;
  bool nt_w;
};
GroupedPlan grouped_plan(int64_t n_pairs, int E, bool gate_up);
hipError_t launch_gemm_grouped(const void* A, int lda, const void* W, int64_t w_stride, int ldw,
                               void* C, int ldc, int N, int K, int epi, const int32_t* g_off,
                               const int32_t* g_cnt, const int32_t* mtiles, const int32_t* n_mtiles,
                               const int32_t* arow, GroupedPlan plan, bool packed_w, hipStream_t st);
// Reorder a row-major bf16 [rows][K] matrix in place into the strip layout
// (rows % 16 == 0, K % 32 == 0, 16*K*2 bytes <= 160 KiB): N/16 strips of 16
// rows; strip g holds K/32 blocks of 64 lanes x 8 bf16, lane l of block s
// holding row 16g + l%16, columns 32s + 8(l/16) .. +8 (the MFMA B operand).
hipError_t launch_pack_strips(void* W, int64_t rows, int K, hipStream_t st);

// ---- attention (k_attn.hip)
size_t attn_workspace_bytes(int n_rows, int hq, int hkv, int hd, int max_ctx);
// ctx(r) = ctx_len ? ctx_len[r] : (ctx_mod ? r % ctx_mod : 0) + ctx_base
hipError_t launch_attention(const void* q, const void* k_pool, const void* v_pool,
                            int64_t n_pages, const int32_t* page_table, int pt_stride,
                            const int32_t* row_pt, const int32_t* ctx_len, int ctx_mod,
                            int ctx_base, int n_rows, int hq, int hkv, int hd, int max_ctx,
                            bool bf16, void* out, void* ws, size_t ws_bytes, hipStream_t st,
                            hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
// Shared-prefix decode attention (bf16): every row has context ctx; row r
// uses page-table row row_traj[r] (clamped into [0, pt_rows) when pt_rows >
// 0); consecutive rows of one group (row_traj[r] / m) share their first
// prefix_pages pages.  build_groups: derive the group table from row_traj
// (else reuse the one in ws from an earlier call with the same rows); the
// group count is also written to *n_groups_out when given.  Requires
// ctx > 16 * prefix_pages.
size_t attn_shared_workspace_bytes(int n_rows, int hq, int hkv, int hd, int ctx, int prefix_pages);
hipError_t launch_attention_shared(const void* q, const void* k_pool, const void* v_pool,
                                   int64_t n_pages, const int32_t* page_table, int pt_stride,
                                   const int32_t* row_traj, int pt_rows, int m, int prefix_pages,
                                   bool build_groups, int ctx, int n_rows, int hq, int hkv, int hd,
                                   void* out, void* ws,
                                   size_t ws_bytes, hipStream_t st, hipEvent_t ev0 = nullptr,
                                   hipEvent_t ev1 = nullptr, int32_t* n_groups_out = nullptr);

// ---- sampler (k_sample.hip)
struct SampleArgs {
  const void* logits; int n_rows; int vocab; bool bf16; uint64_t seed; float temperature;
  const int32_t* row_logit;   // row r reads logits row row_logit[r], else traj[r] / logit_div, else r
  int logit_div;
  const int32_t* traj;        // [n_rows] trajectory id (counter word 1 is traj + traj_base)
  int traj_base;
  const int32_t* step;        // NULL: use per-trajectory gen count (stateful)
  const int32_t* force;       // NULL or indexed by row (stateless) / by traj (stateful)
  int32_t* token_out; int32_t* sampled_out; float* logprob_out; float* entropy_out;
  // stateful termination (all NULL for the stateless sampler)
  int32_t* gen; float* sum_lp; uint8_t* status; int32_t* last_tok; const int32_t* forced_len;
  uint8_t* finished_out; int32_t* traj_out; int cap; int eos;
  int64_t* tokens_counter;
  int32_t* hist_tok; float* hist_lp;   // NULL or [n_traj][cap]: token t of trajectory g at g*cap + t
  // NULL: one block per row.  Otherwise room for part_cap partials: rows are
  // split into sample_parts(n_rows, vocab) vocabulary slices, one block each,
  // merged by a finalize kernel (set by the launcher; parts 1 without room)
  struct SamplePart* part_out; int64_t part_cap;
  int parts;
};
struct SamplePart {
  float m, s, t;   // softmax state of the slice: max, sum e^(z-m), sum e^(z-m)(z-m)
  float v; int i;  // its Gumbel-max winner (exact score, index)
};
// slices per row: about kSampleBlocks blocks in all, each slice at least
// kSampleMinGroups groups of 4 logits, at most kSampleMaxParts per row, so
// n_rows * parts <= kSampleBlocks + n_rows
constexpr int kSampleBlocks = 1024, kSampleMinGroups = 512, kSampleMaxParts = 128;
int sample_parts(int n_rows, int vocab);
hipError_t launch_sample(const SampleArgs& a, hipStream_t st);
hipError_t launch_gumbel_map(const float* u, float* g, int64_t n, bool fast, hipStream_t st);
float gumbel_fast_bound();   // the fast map's distance bound the sampler's filter assumes

// ---- selection / pages (k_select.hip)
struct GroupArgs {
  uint8_t* status; const int32_t* len; const float* sum_lp; const float* mean_lp;
  int n_groups; int m; int k; int L; int m_up; int early_stop; int step;
  int32_t* kept; uint8_t* complete;
  // page reclaim (page_off NULL: none): trajectory g owns pages[page_off[g] ..
  // page_off[g+1]); the pages of every member of each group that completes
  // are written to free_out in group, member and list order, their number to
  // *n_free; work holds n_groups + 1 ints of scratch (per-group offsets)
  const int32_t* page_off; const int32_t* pages; int32_t* free_out; int32_t* n_free; int32_t* work;
};
hipError_t launch_select(const GroupArgs& a, hipStream_t st);
struct PruneArgs {
  uint8_t* status; const int32_t* gen; const float* sum_lp; uint8_t* freed; int32_t* refcnt;
  uint8_t* group_done; int32_t* done_step; int32_t* kept;
  int n_groups, m, k, L, m_up, early_stop, step;
  const int32_t* grp_m;   // [n_groups] candidates of each group (members j < grp_m[i] exist)
  const int32_t* page_table; int pt_stride; int prompt_pages;
  int32_t* free_stack; int32_t* free_top;     // free_top: device counter
  int n_pages;                                // stack capacity
  int32_t* grp_cnt; int32_t* grp_rel; int32_t* trj_cnt;   // scratch [n_groups] x2, [n_groups*m]
  const int32_t* live_in; int n_live_in; int32_t* live_out;
  int32_t* info;    // out: [0] n_live, [1] n_done, [2] free_top
};
hipError_t launch_prune(const PruneArgs& a, hipStream_t st);
struct StreamArgs {
  const int32_t* gen; const uint8_t* status; int32_t* streamed; uint8_t* fin_sent;
  const int32_t* hist_tok; const float* hist_lp; int cap; int n_traj;
  int64_t threshold; int flush;
  int32_t* desc;        // [n_traj][4] out: traj, start, count, final status (0: more to come)
  int32_t* off;         // [n_traj] scratch: token offset of each descriptor
  int32_t* tok_out; float* lp_out; int64_t out_cap;
  int32_t* info;        // out: [0] descriptors (-1: output capacity exceeded), [1] tokens
};
hipError_t launch_stream(const StreamArgs& a, hipStream_t st);
hipError_t launch_advantages(const int32_t* kept, int n_groups, int k, const float* reward,
                             int n_traj, float eps, float* adv, hipStream_t st);
hipError_t launch_alloc_pages(const int32_t* live, int n_live, const int32_t* gen, int prompt_pages,
                              int32_t* page_table, int pt_stride, int32_t* free_stack,
                              int32_t* free_top, int32_t* info, hipStream_t st);
hipError_t launch_prefill_pages(int n_prompts, int m, const int32_t* grp_m, int prompt_pages,
                                int32_t* page_table,
                                int pt_stride, int32_t* free_stack, int32_t* free_top,
                                int32_t* refcnt, hipStream_t st);

// ---- MoE FFN (k_moe.hip): x += sum over the top-k experts of w_e * expert_e(xn)
struct MoeArgs {
  bf16_t* xn;               // in: RMSNorm(x) (bf16); out: RMSNorm of the updated x when *normed
  float* x; int n_rows, d, E, k, Fe;
  float eps;
  int E_pad;                // router rows padded to a multiple of 128 (zero rows)
  const bf16_t* w_router;   // [E_pad][d]
  float* logits;            // [n_rows][E_pad] router logits
  void* gemm_ws; size_t gemm_ws_bytes;   // workspace of the router GEMM
  const bf16_t* w_gu;       // [E][2Fe][d], gate/up rows interleaved in groups of 16, strip-packed
  const bf16_t* w_down;     // [E][d][Fe]
  int32_t* topk_id; float* topk_w; int32_t* pos_of;            // [n_rows*k]
  int32_t* row_of;          // [n_rows*k]: input row of each expert-sorted position
  int32_t* counts; int32_t* offsets; int32_t* cursors;         // [E]
  int32_t* mtiles;          // [n_rows*k / kGroupedTileRowsMin + E] non-empty expert row tiles
  int32_t* n_mtiles;        // [1]
  int32_t* mtiles_dn;       // the same for the down projection's row tiles
  int32_t* n_mtiles_dn;     // [1]
  bf16_t* h_perm; bf16_t* y_perm;                              // [n_rows*k][Fe | d]
  // Verification of the routing (all NULL in normal use).  Row r has key
  // route_key[r] (NULL: r); each pointer addresses this layer's k entries of
  // key 0, keys dbg_stride elements apart.
  const int32_t* route_key;
  const int32_t* force_ids;  // k expert ids to combine instead of the router's own
                             // choice (entry 0 < 0, or any id outside [0, E): own choice)
  int32_t* own_ids_out;      // the router's own top-k ids, rank order
  float* used_p_out;         // softmax probability of each combined expert
  int64_t dbg_stride;
  // Timing (NULL in normal use): events recorded around the grouped gate/up
  // and down GEMMs, and the number of experts that received rows.
  hipEvent_t ev_gu0, ev_gu1, ev_down0, ev_down1;
  int32_t* touched_out;
};
// *normed: the combine also wrote xn = bf16(RMSNorm(x)) (d <= 4096)
hipError_t launch_moe_ffn(const MoeArgs& a, hipStream_t st, bool* normed);

}  // namespace darts
