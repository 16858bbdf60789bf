// Internal interface between the host library (pced_api.cpp) and the gfx950
// kernels (pced_kernels.hip). Not installed; the public ABI is include/pced.h.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pced {

constexpr int kPage = 16;          // tokens per KV page (= MFMA M/K tile edge)
constexpr int kMaxGroup = 16;      // q-heads per kv-head (MFMA N edge)
constexpr int kFuseBlock = 256;    // threads of the fuse work-groups
constexpr int kFuseInlineQueries = 32;  // queries whose row offsets the fuse gets in its kernel arguments
constexpr int kBetaChunk = 4096;   // vocab entries per beta work-group
constexpr int kLmRowsPad = 48;     // hidden-state rows are padded to a multiple of this
constexpr int kLmRowsMTW = 9;      // many-row LM head: row tiles per wave (up to 32 * 9 = 288 rows at once)
constexpr int kMaxSplitPages = 64; // pages per attention chunk (one page id per lane)
constexpr int kMaxSeg = 8;         // sequences one attention chunk may span
constexpr int kStageUnits = 4;     // 16-byte q units per lane staged in LDS for a chunk's later sequences
// Packed LM-head tiles ordered [64-wide k step][16-row vocab block]: at every k
// step the waves of a launch read adjacent tiles, so the weight stream sweeps W
// as one front (the fastest HBM read pattern measured) instead of one region per
// wave ([vocab block][k step]).
constexpr bool kLmKMajor = true;
// The decoder projections' packed matrices in the same k-step-major order:
// [64-wide k step][16-column tile], so the blocks working on one K slice read
// adjacent tiles at every step.
constexpr bool kProjKMajor = true;

// Element offsets inside a bf16 KV tile (16 tokens x head_dim; see pced.h, pool
// layout): every matrix-core operand of the attention is one contiguous 16-byte
// load per lane. K token t, dim d: the A operand of the 16x16x32 q.k product;
// V: the A operand of the 16x16x16 V^T.P^T product. Used by the kernels and by
// the host-side loading of caches held in host memory.
__host__ __device__ inline int kswz(int t, int d) {
  return ((d >> 5) * 64 + t + 16 * ((d & 31) >> 3)) * 8 + (d & 7);
}
__host__ __device__ inline int vswz(int t, int d) {
  const int j = d >> 4;
  return (((j >> 1) * 64 + (d & 15) + 16 * (t >> 2)) * 2 + (j & 1)) * 4 + (t & 3);
}

// Per-step attention launch arguments (one launch per layer).
struct AttnArgs {
  const void* q;            // [S][L][Hq][D]
  const void* kpool;        // [L][max_pages][Hkv][tile]
  const void* vpool;
  const int32_t* len0;      // [S] lengths at load
  const int32_t* page_table;// [S][maxpps]
  // Balanced plan of the step (written by the planning blocks of the append
  // launch): the pages of all sequences, concatenated in sequence order, are cut
  // into C chunks of equal size (+-1 page); one wave per (chunk, kv-head). A
  // chunk meets up to kMaxSeg sequences ("segments"); each segment yields one
  // partial state of its sequence, or the final output when the sequence lies
  // in a single chunk.
  const int2* chunk_info;   // [C] (segments, pages) of each chunk
  const int4* seg;          // [C][kMaxSeg][2]: {s, first page in chunk, page offset in s - first page,
                            //  token end in this chunk}, {partial index in s, partials of s, tokens of s, 0}
  const int32_t* nparts;    // [S] partial states of each sequence (chunks it meets)
  const int32_t* work_pages;// [C][kMaxSplitPages] physical pages of each chunk
  float* part_acc;          // [S*Hkv][split_stride][G][D] partial outputs (bf16 path: normalised, as bf16)
  float* part_ml;           // [S*Hkv][split_stride][G][2] (running max in log2 units, sum)
  void* x_out;              // [S][Hq*D] layer output, storage type
  float* attn_out;          // optional [S][L][Hq][D]
  float* hidden_out;        // optional [S][Hq*D] (last layer only)
  // bf16 decode attention only, optional: the previous layer's partial states
  // (same plan, [S*Hkv][split_stride][G][D] bf16 and [S*Hkv][split_stride][G][2]),
  // merged by this launch into x_out (and attn_out at layer mrg_layer)
  const uint16_t* mrg_acc;
  const float* mrg_ml;
  int mrg_layer;
  int n_seqs, n_layers, layer, n_q_heads, n_kv_heads, group;
  int max_pages, maxpps, t, split_stride, is_last_layer;
  int kv_reread;            // pages are read by several rows of the launch (prefill): plain loads
  // prefill only: each item of the plan is a group of tq suffix tokens of one
  // sequence (tq_T tokens per sequence in the chunk, rows s * tq_T + i), and
  // `group` counts its tq x (Hq / Hkv) query columns per kv-head
  int tq, tq_T;
  float scale_log2;         // log2(e) / sqrt(D)
};

struct AppendArgs {
  const void* k_new;        // [S][L][Hkv][D]
  const void* v_new;
  void* kpool;
  void* vpool;
  const int32_t* len0;
  const int32_t* page_table;
  int2* chunk_info;         // plan outputs, see AttnArgs
  int4* seg;
  int32_t* nparts;
  int32_t* work_pages;
  int n_seqs, n_layers, n_kv_heads, head_dim, max_pages, maxpps, t;
  int n_chunks, total_pages;  // C and P of the balanced plan (P = pages after the append)
  // Planned pages per sequence are at least min_pages (0, 1: none): the pages
  // past a sequence's own read its last page again and are masked.
  int min_pages;
};

struct LoadArgs {
  const uint64_t* src_k;    // [S] device pointers to [L][len][Hkv][D]
  const uint64_t* src_v;
  const int32_t* items;     // [n_items][2] (sequence, logical page)
  const int32_t* len0;
  const int32_t* page_table;
  void* kpool;
  void* vpool;
  int n_layers, n_kv_heads, head_dim, max_pages, maxpps;
};

struct LmArgs {
  const void* x;            // [rows_pad][K] storage type, rows >= M zero
  const void* w;            // packed bf16 tiles (see pced_pack_lm_head) or f32 [V][K]
  float* logits;            // [M][V]
  int M, V, K, rms;
  int row_groups;           // >= 1: work-groups per vocab chunk, each taking every R-th 48-row group
  // Fused Eq. 2 epilogue (fuse_part != nullptr, M <= 288, one row group): the
  // logits are not written; every block writes its best two tokens per query
  // (over its vocabulary slice) to fuse_part [B][fuse_nblk][5] for k_fuse_final.
  const int32_t* query_seq0;// [B+1]
  const int32_t* query_exp0;// [B+1]
  const float* beta;        // [sum N]
  const float* prior;       // [sum N]
  const int32_t* exp_seq;   // [sum N] row of each expert (the many-row kernel stages beta and prior by row)
  float* fuse_part;
  int n_queries, fuse_nblk;
  const float* rho_in;      // optional [M] row scales used instead of rms (bf16 kernels)
  float* rho_buf;           // optional [M] scratch: the many-row kernel computes the row scales there first
  void* x_packed;           // optional scratch of ceil(M/16)*16*K bf16 (rounded up to the kernel's tile
                            // count): the many-row kernel's operand-ordered copy of x
  size_t w_vb, w_ks;        // packed W: 16-byte units from one vocab block / 64-wide k step to the next
                            // (set by launch_lmhead from kLmKMajor)
};

struct FuseArgs {
  const float* logits;      // [S][V]
  const int32_t* query_seq0;// [B+1]
  const int32_t* query_exp0;// [B+1]
  const float* beta;        // [sum N]
  const float* prior;       // [sum N] gamma * ln(clip(r)) rounded to fp32
  float* part;              // [B][nblk][5]
  int32_t* tokens_out;      // [B] with stride
  int32_t* prev_tok;        // [B]
  int32_t* winner;          // optional [B]
  float* top1;              // optional [B]
  float* top2;              // optional [B]
  int V, nblk, tok_stride;
  int max_n;                // most experts of any query (load batch of the stand-alone fuse)
  int32_t inl_seq0[kFuseInlineQueries + 1];  // query_seq0 / query_exp0 of the first queries
  int32_t inl_exp0[kFuseInlineQueries + 1];
};

// MoE / PoE aggregation (the alternatives to Eq. 3's max): per-expert
// log-sum-exp of the contrastive logits c_k = (1 + beta_k) s_k - beta_k s_0,
// then per vocabulary slice the aggregated score and its best two tokens.
struct AggArgs {
  const float* logits;      // [S][V]
  const int32_t* query_seq0;// [B+1]
  const int32_t* query_exp0;// [B+1]
  const int32_t* exp_seq;   // [sum N]
  const int32_t* exp_query; // [sum N]
  const float* beta;        // [sum N]
  const float* logw;        // [sum N] log pi_k, pi_k = r_k^gamma / sum_j r_j^gamma within the query
  float* lse_part;          // [sum N][nchunk][2]
  float* lse;               // [sum N]
  float* part;              // [B][nblk][5] slice candidates for k_fuse_final
  int V, nchunk, nblk, product;  // product: 0 = mixture (MoE), 1 = product (PoE)
};

struct BetaArgs {
  const float* logits;      // [S][V]
  const int32_t* query_seq0;
  const int32_t* exp_seq;   // [sum N] sequence of each expert slot
  const int32_t* exp_query; // [sum N] query of each expert slot
  float* lse_part;          // [S][nchunk][2]
  float* jsd_part;          // [sum N][nchunk]
  float* beta;              // [sum N]
  const int32_t* query_exp0;// [B+1] (scalar mode)
  int V, nchunk;
};

struct SynthArgs {
  void* q;                  // [S][L][Hq*D]
  void* k_new;              // [S][L][Hkv*D]
  void* v_new;
  const int32_t* seq_query; // [S]
  const int32_t* prev_tok;  // [B]
  uint64_t seed;
  float value_scale;        // sqrt(3)/65536 rounded to fp32
  int n_layers, qdim, kvdim, t, first_token, use_first, bf16;
};

// Decoder-stack projections of one decode step: out[m][n] = rho_m sum_k x[m][k] W[n][k]
// for the M step rows, W packed in 16-row tiles (k_pack_w_bf16 layout), with an
// epilogue per projection.
enum GemmEpi { kEpiQkv = 0, kEpiResid = 1, kEpiSwiglu = 2 };
constexpr int kProjMaxSplit = 16;  // K slices of a projection (partial buffer sized for this many)
constexpr size_t kProjMaxLds = 150 * 1024;  // staged x slice of a projection block
constexpr int kPrefillRows = 2304;  // (sequence, suffix token) rows of one prefill chunk, at least
constexpr int kPrefillParts = 8;   // attention partial states per prefill row and kv-head
struct GemmArgs {
  const void* w;            // packed tiles of this projection
  const uint16_t* x;        // [M][K] bf16 input rows
  int M, K, n_tiles;        // rows, inner dimension, 16-column output tiles
  int ksplit;               // K slices (blocks per column group)
  float* part;              // [ksplit][M][16 n_tiles] fp32 partial sums
  // row scale rho_m = 1/sqrt(sum_p ss_in[p][m] * inv_norm_dim + eps), or 1 without ss_in
  const float* ss_in;       // [M][ld_ss]: row m's per-16-column sums at m * ld_ss + p, p < ss_parts
  // many-row epilogues (launch_proj_epilogue): [M] scratch that receives the row
  // scales of ss_in once (k_rho), read as rho_in instead of a sum in every block
  float* rho_rows;
  const float* rho_in;
  int ss_parts, ld_ss;
  float inv_norm_dim, eps;
  // kEpiResid: h[m][n] += out; a_out = bf16(h * g_next); ss_out[n / 16][m] = sum of h^2 over the tile
  float* h;                 // [M][hidden]
  uint16_t* a_out;          // [M][hidden]
  const uint16_t* g_next;   // [hidden]
  float* ss_out;            // [rows][ld_ss], ld_ss >= hidden/16
  // kEpiSwiglu: tiles alternate gate / up; act[m][f] = bf16(silu(gate) * up)
  uint16_t* act;            // [M][F]
  int F;
  // kEpiQkv: columns [0, Hq*D) q, then k, then v; RoPE at pos = len0[m] + t;
  // q to q_out, k / v into the paged pool at that position
  uint16_t* q_out;          // [S][L][Hq][D]
  uint16_t* qkv_trace;      // optional [M][Hq*D + 2 Hkv*D]: q, k, v after RoPE as stored (parity tracing)
  uint16_t* kpool;
  uint16_t* vpool;
  const int32_t* len0;
  const int32_t* page_table;
  int layer, n_layers, n_q_heads, n_kv_heads, head_dim, max_pages, maxpps, t;
  double log2_theta;
  // [maxpps * page][head_dim / 2]: (cos, sin) of RoPE angle pos * theta^(-2i/D)
  // for each position and pair i (launch_rope_table)
  const float2* rope;
  int num_cus;              // compute units of the device (choice of the many-row path)
};
struct EmbedArgs {
  const uint16_t* embed;    // [V][hidden]
  const uint16_t* g;        // [hidden] first layer's attention norm weight
  const int32_t* tokens;    // [B] with stride
  const int32_t* seq_query; // [S]
  float* h;                 // [S][hidden]
  uint16_t* a_out;          // [S][hidden] bf16(h * g)
  float* ss_out;            // [rows][ld_ss], ld_ss >= hidden/16
  int hidden, vocab, tok_stride, ld_ss;
};
// Rows of one prefill chunk: row r = s*T + i is sequence s's suffix token i0 + i,
// a virtual sequence over s's pages ending at position len_s + i. With tq > 1
// the rows are token groups instead: row r = s*ceil(T/tq) + j covers tokens
// tq j .. min(tq j + tq, T) - 1 and ends at its last one.
struct PrefillMetaArgs {
  const int32_t* len0;      // [S]
  const int32_t* page_table;// [S][maxpps]
  const int32_t* seq_query; // [S]
  int32_t* len0_out;        // [S*T] len0[s] + i
  int32_t* page_table_out;  // [S*T][maxpps] copy of s's row
  int32_t* tok_map;         // [S*T] index of the row's token in tokens [B][n_tokens] (optional)
  int n_seqs, T, i0, n_tokens, maxpps;
  int tq;                   // >= 1: one output row per group of tq tokens (len0 of its last token)
};
// Copy of tokens [start, start + count) of one sequence and layer out of the pool.
struct ReadCacheArgs {
  const void* kpool;
  const void* vpool;
  const int32_t* page_table;  // device [S][maxpps]
  void* k_out;                // [count][Hkv][D]
  void* v_out;
  int seq, layer, start, count, n_kv_heads, head_dim, max_pages, maxpps, bf16;
};

// Optional timing events attached to the first / last dispatch of a launcher.
struct Timing {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};

// launchers (pced_kernels.hip); each returns hipGetLastError() after the launch
hipError_t launch_fill_i32(int32_t* p, int32_t v, size_t n, hipStream_t st);
hipError_t launch_zero_bytes(void* p, size_t nbytes, hipStream_t st);
hipError_t launch_load(const LoadArgs& a, int n_items, bool bf16, hipStream_t st, const Timing* tm = nullptr);
hipError_t launch_append(const AppendArgs& a, bool bf16, hipStream_t st, const Timing* tm = nullptr);
hipError_t launch_attn(const AttnArgs& a, int n_blocks, int head_dim, bool bf16, hipStream_t st, const Timing* tm = nullptr);
int attn_blocks_per_cu(int head_dim, bool bf16);  // resident one-wave blocks per CU
hipError_t launch_attn_combine(const AttnArgs& a, int head_dim, int max_splits, bool bf16, hipStream_t st, const Timing* tm = nullptr);
hipError_t launch_pack_lm_head(const void* w, void* wp, int V, int K, bool bf16, hipStream_t st);
hipError_t launch_lmhead(const LmArgs& a, bool bf16, hipStream_t st, const Timing* tm = nullptr);
hipError_t launch_beta(const BetaArgs& a, int n_seqs, int n_exp, hipStream_t st, const Timing* tm = nullptr);
// k_fuse (timed by tm) then the per-query merge k_fuse_final (timed by tm_merge)
hipError_t launch_fuse(const FuseArgs& a, int n_queries, hipStream_t st, const Timing* tm = nullptr,
                       const Timing* tm_merge = nullptr);
// vocabulary tokens per work-group of the stand-alone fuse (1024, or 512 for few queries)
int fuse_slice(int V, int n_queries, int num_cus);
hipError_t launch_beta_mean(const BetaArgs& a, int n_queries, hipStream_t st);
hipError_t launch_agg(const AggArgs& a, int n_exp, int n_queries, hipStream_t st, const Timing* tm = nullptr);
// the final per-query merge alone (after an LM head with the fused epilogue)
hipError_t launch_fuse_final(const FuseArgs& a, int n_queries, hipStream_t st, const Timing* tm = nullptr);
// vocabulary slices (blocks) of the fused LM-head epilogue for M rows, or 0 if M rows cannot be fused
int lmhead_fused_nblk(int M, int V);
// 32-row tiles of the many-row LM head for M rows of a bf16 LM head (its packed
// x then holds that many tiles, zero past M), or 0 if another kernel runs
int lmhead_wide_tiles(int M, int V, int K);
constexpr int kLmWideMaxRows = 288;  // rows of the largest many-row tile count
hipError_t launch_synth(const SynthArgs& a, int n_seqs, hipStream_t st, const Timing* tm = nullptr);
hipError_t launch_copy_rows(const void* src, void* dst, size_t nbytes, hipStream_t st);
hipError_t launch_stream_read(const void* src, size_t nbytes, uint32_t* xor_out, int num_cus, hipStream_t st);
// pack a [rows][K] bf16 matrix into 16-row tiles, tile i going to slot i * stride + offset
hipError_t launch_pack_tiles(const void* w, void* wp, int rows, int K, int stride, int offset, int n_tiles,
                             hipStream_t st);
hipError_t launch_gemm(const GemmArgs& a, GemmEpi epi, hipStream_t st, const Timing* tm = nullptr);
// The projection epilogue alone, over products already in a.part as one K
// slice ([M][16 n_tiles] fp32, e.g. from a library GEMM).
hipError_t launch_proj_epilogue(const GemmArgs& a, GemmEpi epi, hipStream_t st, const Timing* tm = nullptr);
int proj_tiles_per_wave(int n_tiles);                // 16-column tiles per wave of a projection block
size_t proj_lds_bytes(int rows, int K, int ksplit);  // LDS of a projection block
hipError_t launch_embed(const EmbedArgs& a, int n_seqs, hipStream_t st, const Timing* tm = nullptr);
hipError_t launch_prefill_meta(const PrefillMetaArgs& a, hipStream_t st);
// rho[m] = 1/sqrt(sum_p ss[p][m] * inv_dim + eps) for m < M
hipError_t launch_read_cache(const ReadCacheArgs& a, hipStream_t st);
// The allocation-free entry point's scratch: a library-owned device array of
// kNoAllocScratchBytes per GPU; out = its address on the current device.
constexpr size_t kNoAllocScratchBytes = (size_t)4 << 20;
hipError_t noalloc_scratch(void** out);
hipError_t launch_rho(const float* ss, int parts, int ld, int M, float inv_dim, float eps, float* rho,
                      hipStream_t st);
// RoPE table of GemmArgs::rope for positions 0 .. positions - 1, in fp64 rounded to fp32
hipError_t launch_rope_table(float2* out, int positions, int head_dim, double log2_theta, hipStream_t st);

}  // namespace pced
