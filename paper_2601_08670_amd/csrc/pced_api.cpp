// Host side of libpced: argument validation, workspace carving, the host mirror
// of sequence lengths and page tables, and the launch sequence of a PCED decode
// step (arXiv 2601.08670, Section 3). See include/pced.h for the contract.
#include "pced.h"

#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "pced_internal.h"

using namespace pced;

namespace {

thread_local std::string g_err;

pced_status fail(pced_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define HIP_OK(expr)                                                               \
  do {                                                                             \
    hipError_t e_ = (expr);                                                        \
    if (e_ != hipSuccess) return fail(PCED_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
size_t esize_of(const pced_config& c) { return c.dtype == PCED_BF16 ? 2 : 4; }
int ceil_div(long a, long b) { return (int)((a + b - 1) / b); }

bool cfg_valid(const pced_config* c, std::string* why) {
  auto bad = [&](const char* m) { if (why) *why = m; return false; };
  if (!c) return bad("cfg is NULL");
  if (c->n_layers < 1) return bad("n_layers < 1");
  if (c->n_kv_heads < 1 || c->n_q_heads < 1 || c->n_q_heads % c->n_kv_heads) return bad("n_q_heads must be a positive multiple of n_kv_heads");
  if (c->n_q_heads / c->n_kv_heads > kMaxGroup) return bad("n_q_heads / n_kv_heads > 16");
  if (c->dtype != PCED_BF16 && c->dtype != PCED_F32) return bad("unknown dtype");
  if (c->dtype == PCED_BF16 && c->head_dim != 64 && c->head_dim != 128) return bad("bf16 needs head_dim 64 or 128");
  if (c->dtype == PCED_F32 && (c->head_dim < 4 || c->head_dim > 128 || c->head_dim % 4)) return bad("f32 needs head_dim in [4,128], a multiple of 4");
  if (c->hidden != c->n_q_heads * c->head_dim) return bad("hidden must equal n_q_heads * head_dim");
  if (c->dtype == PCED_BF16 && c->hidden % 256) return bad("bf16 hidden must be a multiple of 256");
  if (c->vocab < 2) return bad("vocab < 2");
  if (c->page_size != kPage) return bad("page_size must be 16");
  if (c->max_queries < 1) return bad("max_queries < 1");
  if (c->max_seqs < 2) return bad("max_seqs < 2");
  if (c->max_pages < 1 || c->max_pages_per_seq < 1) return bad("max_pages and max_pages_per_seq must be >= 1");
  if (c->norm != PCED_NORM_NONE && c->norm != PCED_NORM_RMS) return bad("unknown norm");
  if (c->max_attn_chunks < 0) return bad("max_attn_chunks must be >= 0");
  if (c->aggregation != PCED_AGG_MAX && c->aggregation != PCED_AGG_MOE && c->aggregation != PCED_AGG_POE)
    return bad("unknown aggregation");
  if (c->beta_scalar != 0 && c->beta_scalar != 1) return bad("beta_scalar must be 0 or 1");
  if (c->ffn_dim < 0) return bad("ffn_dim must be >= 0");
  if (c->ffn_dim > 0) {
    if (c->dtype != PCED_BF16) return bad("the decoder stack (ffn_dim > 0) needs bf16");
    if (c->ffn_dim % 64) return bad("ffn_dim must be a multiple of 64");
    if (c->rope_theta < 2) return bad("rope_theta must be >= 2");
  }
  // 32-bit index guards used by the kernels
  if ((double)c->max_seqs * c->vocab > 2147483647.0) return bad("max_seqs * vocab exceeds 2^31");
  return true;
}

struct Layout {
  size_t len0, page_table, seq_query, query_seq0, query_exp0, exp_seq, exp_query, prior, logw, beta_fixed,
      load_items, src_k, src_v, meta_end;
  size_t chunk_info, seg, nparts, work_pages, prev_tok, beta, part_acc, part_ml, x, logits,
      rho, x_packed, fuse_part, lse_part, jsd_part, agg_lse, syn_q, syn_k, syn_v, dec_h, dec_a, dec_act, dec_ss, dec_rho, dec_part,
      rope, pf_len0, pf_pt, pf_tok, pf_glen0, pf_gpt, pf_nparts, pf_rho, pf_h, pf_a, pf_act, pf_ss, pf_q, pf_x, pf_part_acc, pf_part_ml, pf_proj,
      total;
  int pf_rows;          // rows of one prefill chunk (sequences x suffix tokens)
  size_t pf_proj_cols;  // slices x columns per row of the prefill projection partials
  int rows_pad, nblk_fuse, nblk_agg, nchunk, max_work;
  size_t part_slots;
  size_t part_cols;  // slices x columns one row of the projection partial buffer holds
};

Layout make_layout(const pced_config& c) {
  Layout L{};
  const size_t S = c.max_seqs, B = c.max_queries, es = esize_of(c);
  const int G = c.n_q_heads / c.n_kv_heads;
  L.rows_pad = ceil_div(c.max_seqs, kLmRowsPad) * kLmRowsPad;
  L.nblk_fuse = ceil_div(c.vocab, 512);  // at most: the stand-alone fuse's slices are 512 or 1024 tokens
  L.nblk_agg = ceil_div(c.vocab, kFuseBlock);
  L.nchunk = ceil_div(c.vocab, kBetaChunk);
  // every attention chunk holds at least one page: chunks <= pages in use (a
  // prefill chunk's rows count their shared pages once per row)
  L.max_work = c.max_pages;
  if (c.ffn_dim > 0)
    L.max_work = std::max<long>(L.max_work, (long)std::max(c.max_seqs, kPrefillRows) * c.max_pages_per_seq);
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t r = o; o = align_up(o + bytes); return r; };
  // metadata block, uploaded by one copy at load
  L.len0 = take(S * 4);
  L.page_table = take(S * c.max_pages_per_seq * 4);
  L.seq_query = take(S * 4);
  L.query_seq0 = take((B + 1) * 4);
  L.query_exp0 = take((B + 1) * 4);
  L.exp_seq = take(S * 4);
  L.exp_query = take(S * 4);
  L.prior = take(S * 4);
  L.logw = take(S * 4);
  L.beta_fixed = take(S * 4);
  L.load_items = take((size_t)c.max_pages * 2 * 4);
  L.src_k = take(S * 8);
  L.src_v = take(S * 8);
  L.meta_end = o;
  L.chunk_info = take((size_t)L.max_work * 8);
  L.seg = take((size_t)L.max_work * kMaxSeg * 2 * 16);
  L.nparts = take(S * 4);
  L.work_pages = take((size_t)L.max_work * kMaxSplitPages * 4);
  L.prev_tok = take(B * 4);
  L.beta = take(S * 4);
  // split partials: [S*Hkv][stride][G][D] with stride <= pages per sequence.
  // The decode step alternates two sets by layer parity (bf16: both fit the
  // fp32-sized accumulator buffer), so that a layer's attention launch can merge
  // the previous layer's partials while writing its own.
  L.part_slots = (size_t)c.max_seqs * c.n_kv_heads * c.max_pages_per_seq;
  L.part_acc = take(L.part_slots * G * c.head_dim * 4);
  L.part_ml = take(2 * L.part_slots * G * 2 * 4);
  L.x = take((size_t)L.rows_pad * c.hidden * es);
  L.logits = take(S * c.vocab * 4);
  L.rho = take((size_t)L.rows_pad * 4);
  // the many-row LM head's operand-ordered copy of x (bf16, more than 48 rows)
  const bool wide = c.dtype == PCED_BF16 && c.max_seqs > kLmRowsPad;
  L.x_packed = take(wide ? (size_t)kLmWideMaxRows * c.hidden * 2 : 0);
  // per-slice candidates: k_fuse uses 256-column slices, the fused LM-head epilogue 128-column ones
  L.fuse_part = take(B * (size_t)ceil_div(c.vocab, 128) * 5 * 4);
  L.lse_part = take(S * L.nchunk * 2 * 4);
  L.jsd_part = take(S * L.nchunk * 4);
  L.agg_lse = take(S * 4);
  L.syn_q = take(S * c.n_layers * c.n_q_heads * c.head_dim * es);
  L.syn_k = take(S * c.n_layers * c.n_kv_heads * c.head_dim * es);
  L.syn_v = take(S * c.n_layers * c.n_kv_heads * c.head_dim * es);
  // decoder stack (ffn_dim > 0): residual stream, next projection's bf16 input
  // (padded rows: it is also the LM head's x), MLP activation, per-16-column
  // sums of h^2 and the final row scales; the attention's query buffer is syn_q
  const size_t dec = c.ffn_dim > 0 ? 1 : 0;
  L.dec_h = take(dec * S * c.hidden * 4);
  L.dec_a = take(dec * L.rows_pad * c.hidden * 2);
  L.dec_act = take(dec * S * c.ffn_dim * 2);
  L.dec_ss = take(dec * (c.hidden / 16) * S * 4);
  L.dec_rho = take(dec * S * 4);
  // RoPE (cos, sin) per position and pair, written by pced_load_caches
  L.rope = take(dec * (size_t)c.max_pages_per_seq * kPage * (c.head_dim / 2) * 8);
  // K-slice partial sums of a projection: [slices][S][columns]
  L.part_cols = (size_t)kProjMaxSplit *
                std::max<size_t>({(size_t)(c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim, (size_t)c.hidden,
                                  (size_t)c.ffn_dim});
  L.dec_part = take(dec * S * L.part_cols * 4);
  // prefill chunk (ffn_dim > 0): up to pf_rows (sequence, suffix token) rows per pass
  // (a multiple of 16 rows: the many-row projection path reads whole 16-row tiles)
  L.pf_rows = dec ? (int)ceil_div(std::max(c.max_seqs, kPrefillRows), 16) * 16 : 0;
  const size_t PR = L.pf_rows;
  // projection products of a chunk: one slice of up to max_cols columns for
  // more than 48 rows (library GEMM), the split-K slices for up to 48
  const size_t max_cols = std::max<size_t>({(size_t)(c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim,
                                            (size_t)c.hidden, 2 * (size_t)c.ffn_dim});
  L.pf_proj_cols = max_cols;
  L.pf_len0 = take(PR * 4);
  L.pf_pt = take(PR * c.max_pages_per_seq * 4);
  L.pf_tok = take(PR * 4);
  // the attention's token groups (at most one per row)
  L.pf_glen0 = take(PR * 4);
  L.pf_gpt = take(PR * c.max_pages_per_seq * 4);
  L.pf_nparts = take(PR * 4);
  L.pf_rho = take(PR * 4);
  L.pf_h = take(PR * c.hidden * 4);
  L.pf_a = take(PR * c.hidden * 2);
  L.pf_act = take(PR * c.ffn_dim * 2);
  L.pf_ss = take((c.hidden / 16) * PR * 4);
  L.pf_q = take(PR * c.n_q_heads * c.head_dim * 2);
  L.pf_x = take(PR * c.hidden * 2);
  L.pf_part_acc = take(PR * c.n_kv_heads * kPrefillParts * G * c.head_dim * 4);
  L.pf_part_ml = take(PR * c.n_kv_heads * kPrefillParts * G * 2 * 4);
  L.pf_proj = take(std::max(PR * max_cols, (size_t)kLmRowsPad * L.part_cols) * 4);
  L.total = o;
  return L;
}

struct ProfRec {
  int cls;
  hipEvent_t a, b;
  double bytes, flops;
};

}  // namespace

struct pced_ctx {
  pced_config cfg;
  Layout lay;
  char* ws;
  bool bf16;
  int G;
  // host mirror of the loaded batch
  bool loaded = false;
  int B = 0, S = 0, NE = 0;
  std::vector<int32_t> n_experts, seq_off, exp_off, len, page_table;
  bool dynamic_beta = false, beta_frozen = false;
  int t = 0;
  void* kpool = nullptr;
  void* vpool = nullptr;
  std::vector<char> staging;
  int num_cus = 0;
  int attn_waves_per_cu = 8;
  // profiling
  bool prof = false;
  std::vector<ProfRec> recs;
  std::vector<hipEvent_t> ev_free;
  rocblas_handle blas = nullptr;  // created at the first many-row projection
  pced_profile totals{};

  template <class T> T* at(size_t off) { return reinterpret_cast<T*>(ws + off); }
};

namespace {

// Start/stop events of one kernel class launch when profiling is on. They are
// handed to the launcher, which attaches them to the dispatch itself
// (hipExtLaunchKernelGGL), so they time the kernels and not the queue.
struct ProfScope {
  pced_ctx* c;
  ProfRec rec;
  Timing tm;
  bool on;
  ProfScope(pced_ctx* ctx, int cls, double bytes, double flops) : c(ctx), on(ctx->prof) {
    if (!on) return;
    rec.cls = cls;
    rec.bytes = bytes;
    rec.flops = flops;
    rec.a = take();
    rec.b = take();
    if (!rec.a || !rec.b) {  // no events to be had: this launch goes untimed
      if (rec.a) c->ev_free.push_back(rec.a);
      if (rec.b) c->ev_free.push_back(rec.b);
      on = false;
      return;
    }
    tm.start = rec.a;
    tm.stop = rec.b;
  }
  const Timing* timing() const { return on ? &tm : nullptr; }
  hipEvent_t take() {
    if (!c->ev_free.empty()) { hipEvent_t e = c->ev_free.back(); c->ev_free.pop_back(); return e; }
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    return e;
  }
  ~ProfScope() {
    if (on) c->recs.push_back(rec);
  }
};

int device_cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 256;
  return n;
}

// Balanced attention plan for the coming step (lengths after its append): the
// P pages of all sequences, concatenated in sequence order, are cut into C
// chunks of floor(P/C) or ceil(P/C) pages, one wave per (chunk, kv-head). The
// device planner uses the same chunk bounds (chunk c starts at floor(c P / C)).
struct AttnPlan {
  long pages = 0;     // P
  int chunks = 0;     // C
  int max_seg = 0;    // most sequences met by one chunk
  int max_parts = 0;  // most chunks met by one sequence (partial slots per sequence)
  int min_pages = 1;  // planned pages per sequence at least (padding pages are masked)
};

void plan_stats(const std::vector<long>& pre, long P, long C, AttnPlan* out) {
  const int S = (int)pre.size() - 1;
  auto lo = [&](long c) { return c * P / C; };
  auto chunk_of = [&](long u) { return (long)(((u + 1) * C - 1) / P); };
  int max_seg = 0, max_parts = 0;
  int s = 0;
  for (long c = 0; c < C; ++c) {
    const long b = lo(c), e = lo(c + 1);
    while (pre[s + 1] <= b) ++s;  // first sequence of the chunk
    int n = 0;
    for (int r = s; r < S && pre[r] < e; ++r) ++n;
    max_seg = std::max(max_seg, n);
  }
  for (int r = 0; r < S; ++r)
    max_parts = std::max(max_parts, (int)(chunk_of(pre[r + 1] - 1) - chunk_of(pre[r]) + 1));
  out->pages = P;
  out->chunks = (int)C;
  out->max_seg = max_seg;
  out->max_parts = max_parts;
}

// C is the number of chunks whose waves all fit on the chip at once (so every
// wave starts in the first round and streams the same number of pages), at
// least P/64 (one page id per lane), raised when a chunk would meet more
// sequences than a wave can stage q rows for.
AttnPlan plan_for_lengths(const pced_ctx* c, const std::vector<int>& lens, int group = 0, bool pad = false);

AttnPlan plan_attention(const pced_ctx* c) {
  return plan_for_lengths(c, std::vector<int>(c->len.begin(), c->len.end()));
}

// The same plan for rows of the given lengths (before the step's append);
// group: query columns per kv-head of an item (0: the model's q-heads per kv-head).
// pad: every item counts at least the chunk length of the unconstrained plan
// (at most kMaxSplitPages / 2 pages), so that a run of short items does not
// force small chunks when a wave can stage few segments.
AttnPlan plan_for_lengths(const pced_ctx* c, const std::vector<int>& lens, int group, bool pad) {
  const int S = (int)lens.size();
  long cap = std::max<long>(1, (long)c->num_cus * c->attn_waves_per_cu / c->cfg.n_kv_heads);
  if (c->cfg.max_attn_chunks > 0) cap = std::min<long>(cap, c->cfg.max_attn_chunks);
  auto first_c = [&](long P) { return std::max<long>(std::min(cap, P), ceil_div(P, (long)kMaxSplitPages)); };
  int min_pages = 1;
  if (pad && S > 0) {
    long P0 = 0;
    for (int s = 0; s < S; ++s) P0 += ceil_div(lens[s] + 1, kPage);
    min_pages = (int)std::min<long>(kMaxSplitPages / 2, ceil_div(P0, first_c(P0)));
  }
  std::vector<long> pre(S + 1, 0);
  for (int s = 0; s < S; ++s) pre[s + 1] = pre[s] + std::max(min_pages, ceil_div(lens[s] + 1, kPage));
  const long P = pre[S];
  long C = first_c(P);
  // bf16: the later segments' q rows of a chunk are staged by its wave in LDS
  const int per_seg_units = (group > 0 ? group : c->G) * c->cfg.head_dim / 8;
  const int seg_limit = c->bf16 ? std::min(kMaxSeg, 1 + 64 * kStageUnits / per_seg_units) : kMaxSeg;
  AttnPlan plan;
  for (;;) {
    plan_stats(pre, P, C, &plan);
    if (plan.max_seg <= seg_limit || C >= P) break;
    C = std::min(P, C + std::max<long>(1, C / 16));
  }
  plan.min_pages = min_pages;
  return plan;
}

// Device memory a kernel can read directly; anything else (pageable or pinned
// host memory) takes the host path of pced_load_caches.
bool is_device_memory(const void* p) {
  hipPointerAttribute_t attr{};
  if (hipPointerGetAttributes(&attr, p) != hipSuccess) {
    (void)hipGetLastError();  // unregistered host memory: clear the sticky error
    return false;
  }
  return attr.type == hipMemoryTypeDevice || attr.type == hipMemoryTypeManaged || attr.isManaged;
}

// Host path of pced_load_caches: sequence s's cache, held in host memory as
// [L][len][Hkv][D], re-laid on the host into the pool's tiles of each of its
// pages (slots past len zero) and copied into the pool with one hipMemcpyAsync
// per run of consecutive physical pages. The staging image is reused once the
// copies out of it have completed (hence the stream synchronisations).
struct HostLoader {
  const pced_config& cfg;
  hipStream_t st;
  size_t es, tile_elems, page_bytes;  // page_bytes: all kv-heads of one page and layer
  std::vector<char> img;
  size_t used = 0;
  HostLoader(const pced_config& c, hipStream_t s)
      : cfg(c), st(s), es(c.dtype == PCED_BF16 ? 2 : 4), tile_elems((size_t)kPage * c.head_dim),
        page_bytes((size_t)c.n_kv_heads * kPage * c.head_dim * (c.dtype == PCED_BF16 ? 2 : 4)) {}

  pced_status flush() {
    if (used) HIP_OK(hipStreamSynchronize(st));
    used = 0;
    return PCED_OK;
  }

  // one (sequence, layer, K or V) image and its copies
  pced_status put(const void* src, int len, int layer, const int32_t* pt, bool is_v, void* pool) {
    const int D = cfg.head_dim, Hkv = cfg.n_kv_heads, np = ceil_div(len, kPage);
    const size_t bytes = (size_t)np * page_bytes;
    if (used + bytes > img.size()) {
      pced_status r = flush();
      if (r != PCED_OK) return r;
      if (bytes > img.size()) img.resize(std::max(bytes, (size_t)64 << 20));
    }
    char* dst = img.data() + used;
    const bool bf16 = cfg.dtype == PCED_BF16;
    for (int p = 0; p < np; ++p)
      for (int g = 0; g < Hkv; ++g) {
        char* tile = dst + ((size_t)p * Hkv + g) * tile_elems * es;
        for (int t = 0; t < kPage; ++t) {
          const int tok = p * kPage + t;
          const size_t row = (((size_t)layer * len + tok) * Hkv + g) * D;
          for (int d = 0; d < D; ++d) {
            if (bf16) {
              const uint16_t v = tok < len ? ((const uint16_t*)src)[row + d] : 0;
              ((uint16_t*)tile)[is_v ? vswz(t, d) : kswz(t, d)] = v;
            } else {
              ((float*)tile)[(size_t)t * D + d] = tok < len ? ((const float*)src)[row + d] : 0.f;
            }
          }
        }
      }
    const size_t layer_off = (size_t)layer * cfg.max_pages * page_bytes;
    for (int p0 = 0; p0 < np;) {
      int p1 = p0 + 1;
      while (p1 < np && pt[p1] == pt[p1 - 1] + 1) ++p1;
      HIP_OK(hipMemcpyAsync((char*)pool + layer_off + (size_t)pt[p0] * page_bytes, dst + (size_t)p0 * page_bytes,
                            (size_t)(p1 - p0) * page_bytes, hipMemcpyHostToDevice, st));
      p0 = p1;
    }
    used += bytes;
    return PCED_OK;
  }
};

pced_status check_ctx(const pced_ctx* c, bool need_loaded) {
  if (!c) return fail(PCED_ERR_INVALID_ARG, "ctx is NULL");
  if (need_loaded && !c->loaded) return fail(PCED_ERR_STATE, "no batch loaded (call pced_load_caches first)");
  return PCED_OK;
}

FuseArgs fuse_args(pced_ctx* c, const float* logits, int32_t* tokens_out, int tok_stride, const pced_step_out* extra,
                   int nblk) {
  FuseArgs f{};
  f.logits = logits;
  f.query_seq0 = c->at<int32_t>(c->lay.query_seq0);
  f.query_exp0 = c->at<int32_t>(c->lay.query_exp0);
  f.beta = c->at<float>(c->lay.beta);
  f.prior = c->at<float>(c->lay.prior);
  f.part = c->at<float>(c->lay.fuse_part);
  f.tokens_out = tokens_out;
  f.prev_tok = c->at<int32_t>(c->lay.prev_tok);
  f.winner = extra ? extra->winner : nullptr;
  f.top1 = extra ? extra->top1 : nullptr;
  f.top2 = extra ? extra->top2 : nullptr;
  f.V = c->cfg.vocab;
  f.nblk = nblk;
  f.max_n = c->n_experts.empty() ? 0 : *std::max_element(c->n_experts.begin(), c->n_experts.end());
  for (int b = 0; b <= std::min(c->B, kFuseInlineQueries); ++b) {
    f.inl_seq0[b] = c->seq_off[b];
    f.inl_exp0[b] = c->exp_off[b];
  }
  f.tok_stride = tok_stride;
  return f;
}

pced_status copy_beta_used(pced_ctx* c, const pced_step_out* extra, hipStream_t st) {
  if (extra && extra->beta_used)
    HIP_OK(hipMemcpyAsync(extra->beta_used, c->at<float>(c->lay.beta), (size_t)c->NE * 4,
                          hipMemcpyDeviceToDevice, st));
  return PCED_OK;
}

// Launch the beta (first step) and fuse kernels over `logits`.
pced_status run_fuse(pced_ctx* c, const float* logits, bool refresh_beta, int32_t* tokens_out,
                     int tok_stride, const pced_step_out* extra, hipStream_t st) {
  const pced_config& cfg = c->cfg;
  if (c->dynamic_beta && refresh_beta) {
    BetaArgs b{};
    b.logits = logits;
    b.query_seq0 = c->at<int32_t>(c->lay.query_seq0);
    b.exp_seq = c->at<int32_t>(c->lay.exp_seq);
    b.exp_query = c->at<int32_t>(c->lay.exp_query);
    b.lse_part = c->at<float>(c->lay.lse_part);
    b.jsd_part = c->at<float>(c->lay.jsd_part);
    b.beta = c->at<float>(c->lay.beta);
    b.V = cfg.vocab;
    b.nchunk = c->lay.nchunk;
    b.query_exp0 = c->at<int32_t>(c->lay.query_exp0);
    ProfScope ps(c, PCED_PROF_BETA, (double)(c->S + 2.0 * c->NE) * cfg.vocab * 4, 0);
    HIP_OK(launch_beta(b, c->S, c->NE, st, ps.timing()));
    if (cfg.beta_scalar) HIP_OK(launch_beta_mean(b, c->B, st));
    c->beta_frozen = true;
  }
  FuseArgs f = fuse_args(c, logits, tokens_out, tok_stride, extra,
                         cfg.aggregation != PCED_AGG_MAX ? c->lay.nblk_agg
                                                         : ceil_div(cfg.vocab, fuse_slice(cfg.vocab, c->B, c->num_cus)));
  if (cfg.aggregation != PCED_AGG_MAX) {
    AggArgs g{};
    g.logits = logits;
    g.query_seq0 = f.query_seq0;
    g.query_exp0 = f.query_exp0;
    g.exp_seq = c->at<int32_t>(c->lay.exp_seq);
    g.exp_query = c->at<int32_t>(c->lay.exp_query);
    g.beta = f.beta;
    g.logw = c->at<float>(c->lay.logw);
    g.lse_part = c->at<float>(c->lay.lse_part);
    g.lse = c->at<float>(c->lay.agg_lse);
    g.part = f.part;
    g.V = cfg.vocab;
    g.nchunk = c->lay.nchunk;
    g.nblk = c->lay.nblk_agg;
    g.product = cfg.aggregation == PCED_AGG_POE;
    {
      ProfScope ps(c, PCED_PROF_FUSE, 2.0 * (c->NE + c->S) * cfg.vocab * 4, 0);
      HIP_OK(launch_agg(g, c->NE, c->B, st, ps.timing()));
    }
    {
      ProfScope ps(c, PCED_PROF_FUSE, (double)c->B * f.nblk * 5 * 4, 0);
      HIP_OK(launch_fuse_final(f, c->B, st, ps.timing()));
    }
    return copy_beta_used(c, extra, st);
  }
  {
    ProfScope ps(c, PCED_PROF_FUSE, (double)c->S * cfg.vocab * 4, 0);
    ProfScope pm(c, PCED_PROF_FUSE_MERGE, (double)c->B * f.nblk * 5 * 4, 0);
    HIP_OK(launch_fuse(f, c->B, st, ps.timing(), pm.timing()));
  }
  return copy_beta_used(c, extra, st);
}

// After an LM head with the fused Eq. 2 epilogue: only the per-query merge of
// its `nblk` slice candidates remains.
pced_status run_fuse_final(pced_ctx* c, int nblk, int32_t* tokens_out, int tok_stride, const pced_step_out* extra,
                           hipStream_t st) {
  FuseArgs f = fuse_args(c, nullptr, tokens_out, tok_stride, extra, nblk);
  {
    ProfScope ps(c, PCED_PROF_FUSE_MERGE, (double)c->B * nblk * 5 * 4, 0);
    HIP_OK(launch_fuse_final(f, c->B, st, ps.timing()));
  }
  return copy_beta_used(c, extra, st);
}

// LM head over M rows of x. With fuse_nblk > 0 the kernel's epilogue applies
// Eq. 2 and leaves per-slice candidates instead of writing the logits.
pced_status run_lmhead(pced_ctx* c, const void* x, int M, const void* w, float* logits, hipStream_t st,
                       int fuse_nblk = 0, const float* rho_in = nullptr) {
  const pced_config& cfg = c->cfg;
  LmArgs a{};
  a.x = x;
  a.w = w;
  a.logits = logits;
  a.M = M;
  a.V = cfg.vocab;
  a.K = cfg.hidden;
  a.rms = cfg.norm == PCED_NORM_RMS;
  a.rho_in = rho_in;
  a.rho_buf = c->at<float>(c->lay.rho);
  a.x_packed = cfg.max_seqs > kLmRowsPad && c->bf16 ? c->at<void>(c->lay.x_packed) : nullptr;
  if (fuse_nblk > 0) {
    a.query_seq0 = c->at<int32_t>(c->lay.query_seq0);
    a.query_exp0 = c->at<int32_t>(c->lay.query_exp0);
    a.beta = c->at<float>(c->lay.beta);
    a.prior = c->at<float>(c->lay.prior);
    a.exp_seq = c->at<int32_t>(c->lay.exp_seq);
    a.fuse_part = c->at<float>(c->lay.fuse_part);
    a.n_queries = c->B;
    a.fuse_nblk = fuse_nblk;
  }
  const double es = (double)esize_of(cfg);
  const double out_bytes = fuse_nblk > 0 ? (double)c->B * fuse_nblk * 5 * 4 : (double)M * cfg.vocab * 4;
  ProfScope ps(c, PCED_PROF_LMHEAD, (double)cfg.vocab * cfg.hidden * es + (double)M * cfg.hidden * es + out_bytes,
               2.0 * M * cfg.vocab * cfg.hidden);
  HIP_OK(launch_lmhead(a, c->bf16, st, ps.timing()));
  return PCED_OK;
}

// LM head and token choice of a step over the S rows of x (rho_in: optional
// row scales). Eq. 2 and the slice argmax run in the LM head's epilogue when
// beta is known (fixed, or frozen after the first step) and the caller wants no
// logits; otherwise the logits are materialised (dynamic beta needs them at the
// first step).
pced_status run_head(pced_ctx* c, const void* x, const float* rho_in, const void* w, int32_t* tokens_out,
                     int tok_stride, const pced_step_out* extra, hipStream_t st) {
  const pced_config& cfg = c->cfg;
  const bool refresh = c->dynamic_beta && !c->beta_frozen;
  const int fused_nblk = (c->bf16 && !refresh && !(extra && extra->logits) && cfg.aggregation == PCED_AGG_MAX)
                             ? lmhead_fused_nblk(c->S, cfg.vocab) : 0;
  pced_status r;
  if (fused_nblk > 0) {
    r = run_lmhead(c, x, c->S, w, nullptr, st, fused_nblk, rho_in);
    if (r != PCED_OK) return r;
    return run_fuse_final(c, fused_nblk, tokens_out, tok_stride, extra, st);
  }
  float* logits = (extra && extra->logits) ? extra->logits : c->at<float>(c->lay.logits);
  r = run_lmhead(c, x, c->S, w, logits, st, 0, rho_in);
  if (r != PCED_OK) return r;
  return run_fuse(c, logits, refresh, tokens_out, tok_stride, extra, st);
}

pced_status check_room(const pced_ctx* c, int n_tokens) {
  const int P = c->cfg.max_pages_per_seq;
  for (int s = 0; s < c->S; ++s) {
    const long last = (long)c->len[s] + n_tokens - 1;
    if (last / kPage >= P) return fail(PCED_ERR_CAPACITY, "sequence %d cannot hold %d more tokens", s, n_tokens);
    for (long p = c->len[s] / kPage; p <= last / kPage; ++p)
      if (c->page_table[(size_t)s * P + p] < 0)
        return fail(PCED_ERR_CAPACITY, "sequence %d cannot hold %d more tokens", s, n_tokens);
  }
  return PCED_OK;
}

// Byte offsets of the decoder-stack weights inside the packed model buffer:
// per layer the two norm weights and the packed QKV (q, k, v tiles
// concatenated), O, gate/up (gate and up tiles alternating) and down
// matrices, then the same four matrices row-major ([out][in], the same row
// order: gate and up in alternating 16-row blocks) for the library GEMMs of
// many-row passes; then the embedding [V][hidden] and the final norm weight.
struct ModelLayout {
  size_t attn_norm, mlp_norm, qkv, o, gu, down, qkv_rm, o_rm, gu_rm, down_rm, layer_bytes;
  size_t embed, final_norm, total;
};

ModelLayout model_layout(const pced_config& c) {
  ModelLayout m{};
  const size_t H = c.hidden, F = c.ffn_dim, qd = (size_t)c.n_q_heads * c.head_dim,
               kd = (size_t)c.n_kv_heads * c.head_dim;
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t r = o; o = align_up(o + bytes); return r; };
  m.attn_norm = take(H * 2);
  m.mlp_norm = take(H * 2);
  m.qkv = take((qd + 2 * kd) * H * 2);
  m.o = take(H * qd * 2);
  m.gu = take(2 * F * H * 2);
  m.down = take(H * F * 2);
  m.qkv_rm = take((qd + 2 * kd) * H * 2);
  m.o_rm = take(H * qd * 2);
  m.gu_rm = take(2 * F * H * 2);
  m.down_rm = take(H * F * 2);
  m.layer_bytes = o;
  o = m.layer_bytes * c.n_layers;
  m.embed = take((size_t)c.vocab * H * 2);
  m.final_norm = take(H * 2);
  m.total = o;
  return m;
}

// Rows of one pass through the decoder stack and the buffers they use. A decode
// step has one row per sequence; a prefill chunk has one row per (sequence,
// suffix token), each a virtual sequence that shares its base sequence's pages
// and ends at its own token (so attention over it is causal by construction).
// The prefill's attention runs on groups of consecutive suffix tokens of one
// sequence instead (the att_* members): one plan item per group, ending at its
// last token, whose tokens take their own query columns and causal ends.
struct FwdRows {
  int M = 0;
  std::vector<int> lens;             // host: length of each row's sequence before its append
  const int32_t* len0 = nullptr;     // device [M]: the row's length minus the step counter t
  const int32_t* page_table = nullptr;  // device [M][max_pages_per_seq]
  const int32_t* tok = nullptr;      // embedding token of row r: tok[tok_map[r] * tok_stride]
  const int32_t* tok_map = nullptr;
  int tok_stride = 1;
  float* h = nullptr;
  uint16_t* a = nullptr;
  uint16_t* act = nullptr;
  float* ss = nullptr;
  int ld_ss = 0;
  uint16_t* q = nullptr;             // attention queries: [M][L][Hq][D] (per_layer_q) or [M][Hq][D]
  bool per_layer_q = true;
  void* x = nullptr;                 // attention output [M][hidden]
  float* part_acc = nullptr;
  float* part_ml = nullptr;
  size_t part_slots = 0;             // (item, kv-head, partial) slots of G columns in the attention partials
  float* proj_part = nullptr;
  size_t proj_cols = 0;              // slices x columns per row of the projection partials
  float* attn_out = nullptr;
  float* rho_rows = nullptr;         // device [M]: the many-row epilogues' row scales
  // The attention's items: the rows (att_tq = 1), or for the prefill groups of
  // att_tq suffix tokens of one sequence (att_T tokens per sequence), each item
  // ending at its last token; the kernels give a group's tokens their own
  // query columns and causal ends.
  int att_n = 0, att_tq = 1, att_T = 1;
  std::vector<int> att_lens;
  const int32_t* att_len0 = nullptr;
  const int32_t* att_pt = nullptr;
  int32_t* att_nparts = nullptr;     // device [att_n]: partial states of each item (the planner's output)
  // optional per-layer traces (decode rows only; see pced_step_out)
  float* resid_trace = nullptr;
  uint16_t* qkv_trace = nullptr;
  uint16_t* act_trace = nullptr;
};

AttnPlan plan_for_lengths(const pced_ctx* c, const std::vector<int>& lens, int group, bool pad);

// One projection of a pass through the stack. Up to 48 rows: the split-K
// kernel on the packed tiles, whose weight stream is the cost. More rows (the
// prefill's chunks): the products are a dense contraction that the split-K
// kernel would stream W for once per 48-row group, so rocBLAS computes them
// (bf16 operands, fp32 accumulation and output) from the row-major copy as a
// single K slice, and the epilogue kernel finishes the projection.
pced_status project(pced_ctx* c, const GemmArgs& g, const char* w_rm, GemmEpi epi, hipStream_t st,
                    const Timing* tm) {
  if (g.M <= kLmRowsPad) {
    HIP_OK(launch_gemm(g, epi, st, tm));
    return PCED_OK;
  }
  if (!c->blas && rocblas_create_handle(&c->blas) != rocblas_status_success) {
    c->blas = nullptr;
    return fail(PCED_ERR_HIP, "rocblas_create_handle failed");
  }
  if (rocblas_set_stream(c->blas, st) != rocblas_status_success) return fail(PCED_ERR_HIP, "rocblas_set_stream failed");
  const int N = 16 * g.n_tiles;
  const float one = 1.0f, zero = 0.0f;
  if (tm && tm->start) HIP_OK(hipEventRecord(tm->start, st));
  // column-major view: part^T [N][M] = (W^T)^T [N][K] x^T [K][M]
  const rocblas_status bs = rocblas_gemm_ex(
      c->blas, rocblas_operation_transpose, rocblas_operation_none, N, g.M, g.K, &one, w_rm, rocblas_datatype_bf16_r,
      g.K, g.x, rocblas_datatype_bf16_r, g.K, &zero, g.part, rocblas_datatype_f32_r, N, g.part, rocblas_datatype_f32_r,
      N, rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
  if (bs != rocblas_status_success) return fail(PCED_ERR_HIP, "rocblas_gemm_ex: %s", rocblas_status_to_string(bs));
  const Timing stop{nullptr, tm ? tm->stop : nullptr};
  HIP_OK(launch_proj_epilogue(g, epi, st, tm ? &stop : nullptr));
  return PCED_OK;
}

// Embedding plus every decoder layer for the rows (appending their K/V rows).
// Leaves the residual stream in rows.h and bf16(h * g_final) in rows.a.
pced_status run_model_forward(pced_ctx* c, const char* model, const FwdRows& R, hipStream_t st) {
  const pced_config& cfg = c->cfg;
  const ModelLayout ml = model_layout(cfg);
  pced_status r = PCED_OK;
  const int M = R.M, H = cfg.hidden, D = cfg.head_dim;
  const int qd = cfg.n_q_heads * D, kd = cfg.n_kv_heads * D;
  const int AG = c->G * R.att_tq;  // query columns per kv-head of an attention item
  const AttnPlan plan = plan_for_lengths(c, R.att_lens, AG, R.att_tq > 1);
  if (plan.chunks > c->lay.max_work) return fail(PCED_ERR_CAPACITY, "attention plan exceeds workspace");
  // (the partial buffers hold part_slots states of G columns)
  if ((size_t)R.att_n * cfg.n_kv_heads * plan.max_parts * AG > R.part_slots * c->G)
    return fail(PCED_ERR_CAPACITY, "attention partial states exceed workspace");
  // per-layer pool offset when the queries are not laid out per layer (the
  // kernels then address layer 0 of the offset pools)
  const size_t layer_elems = (size_t)cfg.max_pages * cfg.n_kv_heads * kPage * D;

  AppendArgs ap{};  // planning blocks only: K/V rows come from the QKV epilogue
  ap.kpool = c->kpool;
  ap.vpool = c->vpool;
  ap.len0 = R.att_len0;
  ap.page_table = R.att_pt;
  ap.chunk_info = c->at<int2>(c->lay.chunk_info);
  ap.seg = c->at<int4>(c->lay.seg);
  ap.nparts = R.att_nparts;
  ap.work_pages = c->at<int32_t>(c->lay.work_pages);
  ap.n_seqs = R.att_n;
  ap.n_layers = cfg.n_layers;
  ap.n_kv_heads = cfg.n_kv_heads;
  ap.head_dim = D;
  ap.max_pages = cfg.max_pages;
  ap.maxpps = cfg.max_pages_per_seq;
  ap.t = c->t;
  ap.n_chunks = plan.chunks;
  ap.total_pages = (int)plan.pages;
  ap.min_pages = plan.min_pages;
  {
    ProfScope ps(c, PCED_PROF_APPEND, 0, 0);
    HIP_OK(launch_append(ap, true, st, ps.timing()));
  }
  {
    EmbedArgs e{};
    e.embed = (const uint16_t*)(model + ml.embed);
    e.g = (const uint16_t*)(model + ml.attn_norm);
    e.tokens = R.tok;
    e.seq_query = R.tok_map;
    e.h = R.h;
    e.a_out = R.a;
    e.ss_out = R.ss;
    e.hidden = H;
    e.vocab = cfg.vocab;
    e.tok_stride = R.tok_stride;
    e.ld_ss = R.ld_ss;
    ProfScope ps(c, PCED_PROF_EMBED, (double)M * H * (2 + 4 + 2), 0);
    HIP_OK(launch_embed(e, M, st, ps.timing()));
  }
  const size_t h_bytes = (size_t)M * H * 4;
  auto trace_h = [&](int l, int j) -> pced_status {  // residual stream entering layer l's block j
    if (R.resid_trace)
      HIP_OK(hipMemcpyAsync(R.resid_trace + ((size_t)l * 2 + j) * M * H, R.h, h_bytes, hipMemcpyDeviceToDevice, st));
    return PCED_OK;
  };
  if (trace_h(0, 0) != PCED_OK) return PCED_ERR_HIP;

  AttnArgs at{};
  at.q = R.q;
  at.len0 = R.att_len0;
  at.page_table = R.att_pt;
  at.chunk_info = ap.chunk_info;
  at.seg = ap.seg;
  at.nparts = R.att_nparts;
  at.work_pages = ap.work_pages;
  at.part_acc = R.part_acc;
  at.part_ml = R.part_ml;
  at.x_out = R.x;
  at.attn_out = R.per_layer_q ? R.attn_out : nullptr;
  at.hidden_out = nullptr;
  at.n_seqs = R.att_n;
  at.n_layers = R.per_layer_q ? cfg.n_layers : 1;
  at.kv_reread = R.per_layer_q ? 0 : 1;  // prefill: the token groups of a sequence share its pages
  at.n_q_heads = cfg.n_q_heads;
  at.n_kv_heads = cfg.n_kv_heads;
  at.group = AG;
  at.tq = R.att_tq;
  at.tq_T = R.att_T;
  at.max_pages = cfg.max_pages;
  at.maxpps = cfg.max_pages_per_seq;
  at.t = c->t;
  at.split_stride = plan.max_parts;
  at.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)D));
  double kv_tokens = 0, kv_item_tokens = 0;  // keys per query row; keys read per item
  for (int r = 0; r < M; ++r) kv_tokens += R.lens[r] + 1;
  for (int v = 0; v < R.att_n; ++v) kv_item_tokens += R.att_lens[v] + 1;
  const double attn_bytes = kv_item_tokens * 2.0 * kd * 2 + 2.0 * M * qd * 2;
  const double attn_flops = kv_tokens * 4.0 * qd;

  GemmArgs g{};
  g.M = M;
  g.ld_ss = R.ld_ss;
  g.ss_parts = H / 16;
  g.inv_norm_dim = 1.0f / (float)H;
  g.eps = 1e-5f;
  g.h = R.h;
  g.a_out = R.a;
  g.ss_out = R.ss;
  g.act = R.act;
  g.F = cfg.ffn_dim;
  g.q_out = R.q;
  g.len0 = R.len0;
  g.page_table = R.page_table;
  g.n_layers = R.per_layer_q ? cfg.n_layers : 1;
  g.n_q_heads = cfg.n_q_heads;
  g.n_kv_heads = cfg.n_kv_heads;
  g.head_dim = D;
  g.max_pages = cfg.max_pages;
  g.maxpps = cfg.max_pages_per_seq;
  g.t = c->t;
  g.log2_theta = std::log2((double)cfg.rope_theta);
  g.rope = c->at<float2>(c->lay.rope);
  g.num_cus = c->num_cus;
  g.part = R.proj_part;
  g.rho_rows = R.rho_rows;
  // K slices per projection: about one block per compute unit, more where the
  // staged x slice would not fit in LDS
  const int stage_rows = std::min(M, M <= 16 ? 16 : M <= 32 ? 32 : 48);
  // (more than 48 rows: one slice, the library GEMM's products)
  auto slices = [&](int n_tiles, int K) {
    if (M > kLmRowsPad) return 1;
    const int groups = ceil_div(n_tiles, 8 * proj_tiles_per_wave(n_tiles));
    int ks = std::max(1, std::min({kProjMaxSplit, K / 64, c->num_cus / groups}));
    while (ks < std::min(kProjMaxSplit, K / 64) && proj_lds_bytes(stage_rows, K, ks) > kProjMaxLds) ++ks;
    return ks;
  };
  auto fits = [&](const GemmArgs& p) {
    return (M > kLmRowsPad || proj_lds_bytes(stage_rows, p.K, p.ksplit) <= kProjMaxLds) &&
           (size_t)p.ksplit * 16 * p.n_tiles <= R.proj_cols;
  };
  const double F = cfg.ffn_dim;
  for (int l = 0; l < cfg.n_layers; ++l) {
    const char* lw = model + (size_t)l * ml.layer_bytes;
    const uint16_t* g_next = (const uint16_t*)(l + 1 < cfg.n_layers ? model + (size_t)(l + 1) * ml.layer_bytes +
                                                                          ml.attn_norm
                                                                    : model + ml.final_norm);
    uint16_t* kp = (uint16_t*)c->kpool;
    uint16_t* vp = (uint16_t*)c->vpool;
    int lq = l;
    if (!R.per_layer_q) {
      kp += (size_t)l * layer_elems;
      vp += (size_t)l * layer_elems;
      lq = 0;
    }
    g.layer = lq;
    g.kpool = kp;
    g.vpool = vp;
    {  // norm + QKV + RoPE + append
      GemmArgs q = g;
      q.w = lw + ml.qkv;
      q.x = R.a;
      q.K = H;
      q.n_tiles = (qd + 2 * kd) / 16;
      q.ksplit = slices(q.n_tiles, H);
      q.ss_in = R.ss;
      q.qkv_trace = R.qkv_trace ? R.qkv_trace + (size_t)l * M * (qd + 2 * kd) : nullptr;
      ProfScope ps(c, PCED_PROF_QKV, (double)(qd + 2 * kd) * H * 2 + (double)M * (H * 2 + (qd + 2 * kd) * 2),
                   2.0 * M * (qd + 2 * kd) * H);
      if (!fits(q)) return fail(PCED_ERR_UNSUPPORTED, "QKV projection does not fit the partial buffer or LDS");
      r = project(c, q, lw + ml.qkv_rm, kEpiQkv, st, ps.timing());
      if (r != PCED_OK) return r;
    }
    at.layer = lq;
    at.kpool = kp;
    at.vpool = vp;
    at.is_last_layer = l == cfg.n_layers - 1;
    {
      ProfScope ps(c, PCED_PROF_ATTN, attn_bytes, attn_flops);
      HIP_OK(launch_attn(at, plan.chunks * cfg.n_kv_heads, D, true, st, ps.timing()));
    }
    if (plan.max_parts > 1) {
      ProfScope ps(c, PCED_PROF_COMBINE, 0, 0);
      HIP_OK(launch_attn_combine(at, D, plan.max_parts, true, st, ps.timing()));
    }
    {  // O projection + residual; the MLP norm's input
      GemmArgs o = g;
      o.w = lw + ml.o;
      o.x = (const uint16_t*)R.x;
      o.K = qd;
      o.n_tiles = H / 16;
      o.ksplit = slices(o.n_tiles, qd);
      o.g_next = (const uint16_t*)(lw + ml.mlp_norm);
      ProfScope ps(c, PCED_PROF_OPROJ, (double)H * qd * 2 + (double)M * (qd * 2 + H * 10), 2.0 * M * H * qd);
      if (!fits(o)) return fail(PCED_ERR_UNSUPPORTED, "O projection does not fit the partial buffer or LDS");
      r = project(c, o, lw + ml.o_rm, kEpiResid, st, ps.timing());
      if (r != PCED_OK) return r;
    }
    if (trace_h(l, 1) != PCED_OK) return PCED_ERR_HIP;
    {  // norm + gate/up + SwiGLU
      GemmArgs u = g;
      u.w = lw + ml.gu;
      u.x = R.a;
      u.K = H;
      u.n_tiles = 2 * cfg.ffn_dim / 16;
      u.ksplit = slices(u.n_tiles, H);
      u.ss_in = R.ss;
      ProfScope ps(c, PCED_PROF_GATEUP, 2.0 * F * H * 2 + (double)M * (H * 2 + F * 2), 4.0 * M * F * H);
      if (!fits(u)) return fail(PCED_ERR_UNSUPPORTED, "gate/up projection does not fit the partial buffer or LDS");
      r = project(c, u, lw + ml.gu_rm, kEpiSwiglu, st, ps.timing());
      if (r != PCED_OK) return r;
    }
    if (R.act_trace)
      HIP_OK(hipMemcpyAsync(R.act_trace + (size_t)l * M * cfg.ffn_dim, R.act, (size_t)M * cfg.ffn_dim * 2,
                            hipMemcpyDeviceToDevice, st));
    {  // down projection + residual; the next norm's input
      GemmArgs d = g;
      d.w = lw + ml.down;
      d.x = R.act;
      d.K = cfg.ffn_dim;
      d.n_tiles = H / 16;
      d.ksplit = slices(d.n_tiles, cfg.ffn_dim);
      d.g_next = g_next;
      ProfScope ps(c, PCED_PROF_DOWN, F * H * 2 + (double)M * (F * 2 + H * 10), 2.0 * M * H * F);
      if (!fits(d)) return fail(PCED_ERR_UNSUPPORTED, "down projection does not fit the partial buffer or LDS");
      r = project(c, d, lw + ml.down_rm, kEpiResid, st, ps.timing());
      if (r != PCED_OK) return r;
    }
    if (l + 1 < cfg.n_layers && trace_h(l + 1, 0) != PCED_OK) return PCED_ERR_HIP;
  }
  return PCED_OK;
}

// The rows of a decode step: one per sequence.
FwdRows decode_rows(pced_ctx* c, const int32_t* in_tok, const pced_step_out* extra) {
  const pced_config& cfg = c->cfg;
  FwdRows R;
  R.M = c->S;
  R.lens.assign(c->len.begin(), c->len.end());
  R.len0 = c->at<int32_t>(c->lay.len0);
  R.page_table = c->at<int32_t>(c->lay.page_table);
  R.att_n = R.M;
  R.att_lens = R.lens;
  R.att_len0 = R.len0;
  R.att_pt = R.page_table;
  R.att_nparts = c->at<int32_t>(c->lay.nparts);
  R.tok = in_tok;
  R.tok_map = c->at<int32_t>(c->lay.seq_query);
  R.tok_stride = 1;
  R.h = c->at<float>(c->lay.dec_h);
  R.a = c->at<uint16_t>(c->lay.dec_a);
  R.act = c->at<uint16_t>(c->lay.dec_act);
  R.ss = c->at<float>(c->lay.dec_ss);
  R.ld_ss = cfg.hidden / 16;
  R.q = c->at<uint16_t>(c->lay.syn_q);
  R.per_layer_q = true;
  R.x = c->at<void>(c->lay.x);
  R.part_acc = c->at<float>(c->lay.part_acc);
  R.part_ml = c->at<float>(c->lay.part_ml);
  R.part_slots = c->lay.part_slots;
  R.rho_rows = c->at<float>(c->lay.dec_rho);  // (the final norm's scales are computed after the layers)
  R.proj_part = c->at<float>(c->lay.dec_part);
  R.proj_cols = c->lay.part_cols;
  if (extra) {
    R.attn_out = extra->attn_out;
    R.resid_trace = extra->resid_trace;
    R.qkv_trace = extra->qkv_trace;
    R.act_trace = extra->act_trace;
  }
  return R;
}

// One chunk of the query-suffix prefill: suffix tokens i0 .. i0+T-1 of every
// query as S*T rows (row s*T + i: sequence s, token i0 + i, position len_s + i).
pced_status run_prefill_chunk(pced_ctx* c, const char* model, const int32_t* tokens, int n_tokens, int i0, int T,
                              hipStream_t st) {
  const pced_config& cfg = c->cfg;
  const int S = c->S, M = S * T;
  PrefillMetaArgs pm{};
  pm.len0 = c->at<int32_t>(c->lay.len0);
  pm.page_table = c->at<int32_t>(c->lay.page_table);
  pm.seq_query = c->at<int32_t>(c->lay.seq_query);
  pm.len0_out = c->at<int32_t>(c->lay.pf_len0);
  pm.page_table_out = c->at<int32_t>(c->lay.pf_pt);
  pm.tok_map = c->at<int32_t>(c->lay.pf_tok);
  pm.n_seqs = S;
  pm.T = T;
  pm.i0 = i0;
  pm.n_tokens = n_tokens;
  pm.maxpps = cfg.max_pages_per_seq;
  pm.tq = 1;
  HIP_OK(launch_prefill_meta(pm, st));
  FwdRows R;
  R.M = M;
  R.lens.resize(M);
  for (int s = 0; s < S; ++s)
    for (int i = 0; i < T; ++i) R.lens[(size_t)s * T + i] = c->len[s] + i;
  R.len0 = pm.len0_out;
  R.page_table = pm.page_table_out;
  // attention items: groups of tq tokens of a sequence fill the matrix cores' 16
  // query columns per kv-head (tq x q-heads per kv-head), so each group reads
  // the sequence's pages once for all its tokens
  // (fewer tokens per group where the partial states of the plan would not fit)
  const size_t part_slots = (size_t)c->lay.pf_rows * cfg.n_kv_heads * kPrefillParts;
  int tq = std::max(1, std::min(T, kMaxGroup / c->G)), ng = 0;
  for (;; tq = (tq + 1) / 2) {
    ng = ceil_div(T, tq);
    R.att_lens.resize((size_t)S * ng);
    for (int s = 0; s < S; ++s)
      for (int j = 0; j < ng; ++j) R.att_lens[(size_t)s * ng + j] = c->len[s] + std::min(tq * j + tq, T) - 1;
    if (tq == 1) break;
    const AttnPlan p = plan_for_lengths(c, R.att_lens, c->G * tq, true);
    if ((size_t)S * ng * cfg.n_kv_heads * p.max_parts * tq <= part_slots) break;
  }
  PrefillMetaArgs gm = pm;
  gm.len0_out = c->at<int32_t>(c->lay.pf_glen0);
  gm.page_table_out = c->at<int32_t>(c->lay.pf_gpt);
  gm.tok_map = nullptr;
  gm.tq = tq;
  HIP_OK(launch_prefill_meta(gm, st));
  R.att_n = S * ng;
  R.att_tq = tq;
  R.att_T = T;
  R.att_len0 = gm.len0_out;
  R.att_pt = gm.page_table_out;
  R.att_nparts = c->at<int32_t>(c->lay.pf_nparts);
  R.tok = tokens;
  R.tok_map = pm.tok_map;
  R.tok_stride = 1;
  R.h = c->at<float>(c->lay.pf_h);
  R.a = c->at<uint16_t>(c->lay.pf_a);
  R.act = c->at<uint16_t>(c->lay.pf_act);
  R.ss = c->at<float>(c->lay.pf_ss);
  R.ld_ss = cfg.hidden / 16;
  R.q = c->at<uint16_t>(c->lay.pf_q);
  R.per_layer_q = false;
  R.x = c->at<void>(c->lay.pf_x);
  R.part_acc = c->at<float>(c->lay.pf_part_acc);
  R.part_ml = c->at<float>(c->lay.pf_part_ml);
  R.part_slots = part_slots;
  R.rho_rows = c->at<float>(c->lay.pf_rho);
  R.proj_part = c->at<float>(c->lay.pf_proj);
  R.proj_cols = M > kLmRowsPad ? c->lay.pf_proj_cols : c->lay.part_cols;
  return run_model_forward(c, model, R, st);
}

pced_status check_model(const pced_ctx* c, const void* model) {
  pced_status r = check_ctx(c, true);
  if (r != PCED_OK) return r;
  if (c->cfg.ffn_dim <= 0) return fail(PCED_ERR_STATE, "no decoder stack configured (ffn_dim == 0)");
  if (!model) return fail(PCED_ERR_INVALID_ARG, "model is NULL");
  return PCED_OK;
}

// One decode step through the decoder stack (shared by step and generate).
pced_status run_model_step(pced_ctx* c, const void* model, const void* w, const int32_t* in_tok, int32_t* tokens_out,
                           int tok_stride, const pced_step_out* extra, hipStream_t st) {
  pced_status r = check_room(c, 1);
  if (r != PCED_OK) return r;
  r = run_model_forward(c, (const char*)model, decode_rows(c, in_tok, extra), st);
  if (r != PCED_OK) return r;
  const pced_config& cfg = c->cfg;
  float* rho = c->at<float>(c->lay.dec_rho);
  HIP_OK(launch_rho(c->at<float>(c->lay.dec_ss), cfg.hidden / 16, cfg.hidden / 16, c->S, 1.0f / (float)cfg.hidden,
                    1e-5f, rho, st));
  r = run_head(c, c->at<void>(c->lay.dec_a), rho, w, tokens_out, tok_stride, extra, st);
  if (r != PCED_OK) return r;
  if (extra && extra->hidden)
    HIP_OK(hipMemcpyAsync(extra->hidden, c->at<float>(c->lay.dec_h), (size_t)c->S * cfg.hidden * 4,
                          hipMemcpyDeviceToDevice, st));
  for (int s = 0; s < c->S; ++s) c->len[s] += 1;
  c->t += 1;
  return PCED_OK;
}

// The step body shared by pced_step and pced_generate.
pced_status run_step(pced_ctx* c, const void* q, const void* k_new, const void* v_new, const void* w,
                     int32_t* tokens_out, int tok_stride, const pced_step_out* extra, hipStream_t st) {
  const pced_config& cfg = c->cfg;
  const int P = cfg.max_pages_per_seq;
  for (int s = 0; s < c->S; ++s) {
    const int pidx = c->len[s] / kPage;
    if (pidx >= P || c->page_table[(size_t)s * P + pidx] < 0)
      return fail(PCED_ERR_CAPACITY, "sequence %d has no page for token %d", s, c->len[s]);
  }
  const AttnPlan plan = plan_attention(c);
  if (plan.chunks > c->lay.max_work) return fail(PCED_ERR_CAPACITY, "attention plan exceeds workspace");
  const double es = (double)esize_of(cfg);

  AppendArgs ap{};
  ap.k_new = k_new;
  ap.v_new = v_new;
  ap.kpool = c->kpool;
  ap.vpool = c->vpool;
  ap.len0 = c->at<int32_t>(c->lay.len0);
  ap.page_table = c->at<int32_t>(c->lay.page_table);
  ap.chunk_info = c->at<int2>(c->lay.chunk_info);
  ap.seg = c->at<int4>(c->lay.seg);
  ap.nparts = c->at<int32_t>(c->lay.nparts);
  ap.work_pages = c->at<int32_t>(c->lay.work_pages);
  ap.n_seqs = c->S;
  ap.n_layers = cfg.n_layers;
  ap.n_kv_heads = cfg.n_kv_heads;
  ap.head_dim = cfg.head_dim;
  ap.max_pages = cfg.max_pages;
  ap.maxpps = P;
  ap.t = c->t;
  ap.n_chunks = plan.chunks;
  ap.total_pages = (int)plan.pages;
  ap.min_pages = plan.min_pages;
  {
    ProfScope ps(c, PCED_PROF_APPEND, 4.0 * c->S * cfg.n_layers * cfg.n_kv_heads * cfg.head_dim * es, 0);
    HIP_OK(launch_append(ap, c->bf16, st, ps.timing()));
  }

  AttnArgs at{};
  at.q = q;
  at.kpool = c->kpool;
  at.vpool = c->vpool;
  at.len0 = ap.len0;
  at.page_table = ap.page_table;
  at.chunk_info = ap.chunk_info;
  at.seg = ap.seg;
  at.nparts = ap.nparts;
  at.work_pages = ap.work_pages;
  at.part_acc = c->at<float>(c->lay.part_acc);
  at.part_ml = c->at<float>(c->lay.part_ml);
  at.x_out = c->at<void>(c->lay.x);
  at.attn_out = extra ? extra->attn_out : nullptr;
  at.hidden_out = extra ? extra->hidden : nullptr;
  at.n_seqs = c->S;
  at.n_layers = cfg.n_layers;
  at.n_q_heads = cfg.n_q_heads;
  at.n_kv_heads = cfg.n_kv_heads;
  at.group = c->G;
  at.max_pages = cfg.max_pages;
  at.maxpps = P;
  at.t = c->t;
  at.split_stride = plan.max_parts;
  at.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)cfg.head_dim));
  double kv_tokens = 0;
  for (int s = 0; s < c->S; ++s) kv_tokens += c->len[s] + 1;
  const double attn_bytes = kv_tokens * 2.0 * cfg.n_kv_heads * cfg.head_dim * es +
                            2.0 * c->S * cfg.n_q_heads * cfg.head_dim * es;
  const double attn_flops = kv_tokens * 4.0 * cfg.n_q_heads * cfg.head_dim;
  // Sequences that span several chunks need a merge of their partial states.
  // bf16: layer l's partials go to set l % 2 and the attention launch of layer
  // l + 1 merges them (one launch per layer instead of two); only the last
  // layer's merge is a launch of its own.
  const bool split = plan.max_parts > 1;
  const bool fold = split && c->bf16;
  const size_t acc_set = c->lay.part_slots * c->G * cfg.head_dim / 2;  // floats per bf16 set
  const size_t ml_set = c->lay.part_slots * c->G * 2;
  float* acc0 = at.part_acc;
  float* ml0 = at.part_ml;
  for (int l = 0; l < cfg.n_layers; ++l) {
    at.layer = l;
    at.is_last_layer = l == cfg.n_layers - 1;
    const int set = fold ? l & 1 : 0;
    at.part_acc = acc0 + set * acc_set;
    at.part_ml = ml0 + set * ml_set;
    const bool merge_prev = fold && l > 0;
    at.mrg_acc = merge_prev ? (const uint16_t*)(acc0 + (set ^ 1) * acc_set) : nullptr;
    at.mrg_ml = merge_prev ? ml0 + (set ^ 1) * ml_set : nullptr;
    at.mrg_layer = l - 1;
    {
      ProfScope ps(c, PCED_PROF_ATTN, attn_bytes, attn_flops);
      HIP_OK(launch_attn(at, plan.chunks * cfg.n_kv_heads, cfg.head_dim, c->bf16, st, ps.timing()));
    }
    if (split && (!fold || l == cfg.n_layers - 1)) {
      ProfScope ps(c, PCED_PROF_COMBINE, 0, 0);
      HIP_OK(launch_attn_combine(at, cfg.head_dim, plan.max_parts, c->bf16, st, ps.timing()));
    }
  }
  at.mrg_acc = nullptr;
  at.mrg_ml = nullptr;

  const pced_status r = run_head(c, at.x_out, nullptr, w, tokens_out, tok_stride, extra, st);
  if (r != PCED_OK) return r;
  for (int s = 0; s < c->S; ++s) c->len[s] += 1;
  c->t += 1;
  return PCED_OK;
}

}  // namespace

extern "C" {

size_t pced_pool_bytes(const pced_config* cfg) {
  if (!cfg_valid(cfg, nullptr)) return 0;
  return (size_t)cfg->n_layers * cfg->max_pages * cfg->n_kv_heads * kPage * cfg->head_dim * esize_of(*cfg);
}

size_t pced_lm_head_bytes(const pced_config* cfg) {
  if (!cfg_valid(cfg, nullptr)) return 0;
  if (cfg->dtype == PCED_BF16) return (size_t)ceil_div(cfg->vocab, 16) * 16 * cfg->hidden * 2;
  return (size_t)cfg->vocab * cfg->hidden * 4;
}

pced_status pced_pack_lm_head(const pced_config* cfg, const void* w, void* w_packed, hipStream_t st) {
  std::string why;
  if (!cfg_valid(cfg, &why)) return fail(PCED_ERR_INVALID_ARG, "invalid config: %s", why.c_str());
  if (!w || !w_packed) return fail(PCED_ERR_INVALID_ARG, "NULL argument");
  const char* a = (const char*)w;
  const char* b = (const char*)w_packed;
  const size_t na = (size_t)cfg->vocab * cfg->hidden * esize_of(*cfg), nb = pced_lm_head_bytes(cfg);
  if (a < b + nb && b < a + na) return fail(PCED_ERR_INVALID_ARG, "w and w_packed overlap");
  HIP_OK(launch_pack_lm_head(w, w_packed, cfg->vocab, cfg->hidden, cfg->dtype == PCED_BF16, st));
  return PCED_OK;
}

size_t pced_workspace_bytes(const pced_config* cfg) {
  if (!cfg_valid(cfg, nullptr)) return 0;
  return make_layout(*cfg).total;
}

const char* pced_last_error(void) { return g_err.c_str(); }

pced_status pced_create(const pced_config* cfg, void* d_workspace, size_t ws_bytes, pced_ctx** out) {
  std::string why;
  if (!out) return fail(PCED_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!cfg_valid(cfg, &why)) return fail(PCED_ERR_INVALID_ARG, "invalid config: %s", why.c_str());
  if (!d_workspace) return fail(PCED_ERR_INVALID_ARG, "workspace is NULL");
  if ((uintptr_t)d_workspace % kAlign) return fail(PCED_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  const Layout lay = make_layout(*cfg);
  if (ws_bytes < lay.total)
    return fail(PCED_ERR_CAPACITY, "workspace too small: %zu < %zu bytes", ws_bytes, lay.total);
  pced_ctx* c = new pced_ctx();
  c->cfg = *cfg;
  c->lay = lay;
  c->ws = (char*)d_workspace;
  c->bf16 = cfg->dtype == PCED_BF16;
  c->G = cfg->n_q_heads / cfg->n_kv_heads;
  *out = c;
  return PCED_OK;
}

void pced_destroy(pced_ctx* ctx) {
  if (!ctx) return;
  for (auto& r : ctx->recs) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  for (auto e : ctx->ev_free) (void)hipEventDestroy(e);
  if (ctx->blas) rocblas_destroy_handle(ctx->blas);
  delete ctx;
}

pced_status pced_load_caches(pced_ctx* c, int32_t n_queries, const int32_t* n_experts,
                             const int32_t* cache_len, const void* const* src_k,
                             const void* const* src_v, void* k_pool, void* v_pool,
                             const int32_t* page_table, int32_t reserve_tokens,
                             const float* relevance, float gamma, const float* beta,
                             hipStream_t st) {
  pced_status r = check_ctx(c, false);
  if (r != PCED_OK) return r;
  const pced_config& cfg = c->cfg;
  if (n_queries < 1 || n_queries > cfg.max_queries)
    return fail(PCED_ERR_INVALID_ARG, "n_queries %d not in [1, %d]", n_queries, cfg.max_queries);
  if (!n_experts || !cache_len || !src_k || !src_v || !k_pool || !v_pool || !relevance)
    return fail(PCED_ERR_INVALID_ARG, "NULL argument");
  if (!std::isfinite(gamma)) return fail(PCED_ERR_INVALID_ARG, "gamma is not finite");
  if (reserve_tokens < 0) return fail(PCED_ERR_INVALID_ARG, "reserve_tokens < 0");
  long S = 0, NE = 0;
  for (int b = 0; b < n_queries; ++b) {
    if (n_experts[b] < 1) return fail(PCED_ERR_INVALID_ARG, "query %d has %d experts", b, n_experts[b]);
    S += n_experts[b] + 1;
    NE += n_experts[b];
  }
  if (S > cfg.max_seqs) return fail(PCED_ERR_CAPACITY, "%ld sequences > max_seqs %d", S, cfg.max_seqs);
  for (long s = 0; s < S; ++s) {
    if (cache_len[s] < 1) return fail(PCED_ERR_INVALID_ARG, "cache_len[%ld] = %d < 1", s, cache_len[s]);
    if (!src_k[s] || !src_v[s]) return fail(PCED_ERR_INVALID_ARG, "source pointer of sequence %ld is NULL", s);
  }
  std::vector<char> on_host(S, 0);
  for (long s = 0; s < S; ++s) {
    const bool dk = is_device_memory(src_k[s]), dv = is_device_memory(src_v[s]);
    if (dk != dv)
      return fail(PCED_ERR_INVALID_ARG, "sequence %ld: src_k and src_v must both be device or both host memory", s);
    on_host[s] = !dk;
  }
  for (long e = 0; e < NE; ++e) {
    if (!std::isfinite(relevance[e])) return fail(PCED_ERR_INVALID_ARG, "relevance[%ld] is not finite", e);
    if (beta && !std::isfinite(beta[e])) return fail(PCED_ERR_INVALID_ARG, "beta[%ld] is not finite", e);
  }
  const int P = cfg.max_pages_per_seq;
  std::vector<int32_t> pt((size_t)S * P, -1);
  if (page_table) {
    std::vector<char> used(cfg.max_pages, 0);
    for (long s = 0; s < S; ++s) {
      const int need = ceil_div(cache_len[s], kPage);
      if (need > P) return fail(PCED_ERR_CAPACITY, "sequence %ld needs %d pages > max_pages_per_seq", s, need);
      for (int p = 0; p < P; ++p) {
        const int32_t id = page_table[s * P + p];
        if (id < 0) {
          if (p < need) return fail(PCED_ERR_INVALID_ARG, "sequence %ld: page %d of its cache not given", s, p);
          continue;
        }
        if (id >= cfg.max_pages) return fail(PCED_ERR_INVALID_ARG, "page id %d >= max_pages", id);
        if (used[id]) return fail(PCED_ERR_INVALID_ARG, "page id %d used twice", id);
        used[id] = 1;
        pt[s * P + p] = id;
      }
    }
  } else {
    long next = 0;
    for (long s = 0; s < S; ++s) {
      const int need = ceil_div((long)cache_len[s] + reserve_tokens, kPage);
      if (need > P) return fail(PCED_ERR_CAPACITY, "sequence %ld needs %d pages > max_pages_per_seq %d", s, need, P);
      if (next + need > cfg.max_pages) return fail(PCED_ERR_CAPACITY, "pool of %d pages exhausted", cfg.max_pages);
      for (int p = 0; p < need; ++p) pt[s * P + p] = (int32_t)(next + p);
      next += need;
    }
  }
  if (c->num_cus == 0) {
    c->num_cus = device_cus();
    c->attn_waves_per_cu = attn_blocks_per_cu(cfg.head_dim, c->bf16);
  }

  // host mirror
  c->B = n_queries;
  c->S = (int)S;
  c->NE = (int)NE;
  c->n_experts.assign(n_experts, n_experts + n_queries);
  c->seq_off.assign(n_queries + 1, 0);
  c->exp_off.assign(n_queries + 1, 0);
  for (int b = 0; b < n_queries; ++b) {
    c->seq_off[b + 1] = c->seq_off[b] + n_experts[b] + 1;
    c->exp_off[b + 1] = c->exp_off[b] + n_experts[b];
  }
  c->len.assign(cache_len, cache_len + S);
  c->page_table = pt;

  // metadata image, uploaded with one copy
  const Layout& L = c->lay;
  c->staging.assign(L.meta_end, 0);
  auto put = [&](size_t off, const void* src, size_t n) { std::memcpy(c->staging.data() + off, src, n); };
  put(L.len0, cache_len, S * 4);
  put(L.page_table, pt.data(), pt.size() * 4);
  std::vector<int32_t> seq_query(S), exp_seq(NE), exp_query(NE);
  std::vector<float> prior(NE), logw(NE), bfix(NE, 0.f);
  std::vector<int32_t> items;
  for (int b = 0; b < n_queries; ++b) {
    for (int k = 0; k <= n_experts[b]; ++k) seq_query[c->seq_off[b] + k] = b;
    for (int k = 1; k <= n_experts[b]; ++k) {
      const int e = c->exp_off[b] + k - 1;
      exp_seq[e] = c->seq_off[b] + k;
      exp_query[e] = b;
      // gamma * ln(r) with r clipped to [1e-8, 1 - 1e-8], in double, rounded once
      const double rr = std::min(std::max((double)relevance[e], 1e-8), 1.0 - 1e-8);
      prior[e] = (float)((double)gamma * std::log(rr));
      if (beta) bfix[e] = beta[e];
    }
    // MoE / PoE weights: log pi_k = gamma ln r_k - log sum_j exp(gamma ln r_j) over the query, in double
    double mx = -INFINITY;
    for (int k = 1; k <= n_experts[b]; ++k) {
      const double rr = std::min(std::max((double)relevance[c->exp_off[b] + k - 1], 1e-8), 1.0 - 1e-8);
      mx = std::max(mx, (double)gamma * std::log(rr));
    }
    double z = 0.0;
    for (int k = 1; k <= n_experts[b]; ++k) {
      const double rr = std::min(std::max((double)relevance[c->exp_off[b] + k - 1], 1e-8), 1.0 - 1e-8);
      z += std::exp((double)gamma * std::log(rr) - mx);
    }
    for (int k = 1; k <= n_experts[b]; ++k) {
      const int e = c->exp_off[b] + k - 1;
      const double rr = std::min(std::max((double)relevance[e], 1e-8), 1.0 - 1e-8);
      logw[e] = (float)((double)gamma * std::log(rr) - mx - std::log(z));
    }
  }
  for (long s = 0; s < S; ++s)
    if (!on_host[s])
      for (int p = 0; p < ceil_div(cache_len[s], kPage); ++p) { items.push_back((int32_t)s); items.push_back(p); }
  put(L.seq_query, seq_query.data(), S * 4);
  put(L.query_seq0, c->seq_off.data(), (n_queries + 1) * 4);
  put(L.query_exp0, c->exp_off.data(), (n_queries + 1) * 4);
  put(L.exp_seq, exp_seq.data(), NE * 4);
  put(L.exp_query, exp_query.data(), NE * 4);
  put(L.prior, prior.data(), NE * 4);
  put(L.logw, logw.data(), NE * 4);
  put(L.beta_fixed, bfix.data(), NE * 4);
  put(L.load_items, items.data(), items.size() * 4);
  std::vector<uint64_t> sk(S), sv(S);
  for (long s = 0; s < S; ++s) { sk[s] = (uint64_t)(uintptr_t)src_k[s]; sv[s] = (uint64_t)(uintptr_t)src_v[s]; }
  put(L.src_k, sk.data(), S * 8);
  put(L.src_v, sv.data(), S * 8);
  HIP_OK(hipMemcpyAsync(c->ws, c->staging.data(), L.meta_end, hipMemcpyHostToDevice, st));

  // per-batch device state
  HIP_OK(launch_fill_i32(c->at<int32_t>(L.prev_tok), -1, cfg.max_queries, st));
  HIP_OK(launch_zero_bytes(c->at<void>(L.x), (size_t)L.rows_pad * cfg.hidden * esize_of(cfg), st));
  if (cfg.ffn_dim > 0)
    HIP_OK(launch_rope_table(c->at<float2>(L.rope), cfg.max_pages_per_seq * kPage, cfg.head_dim,
                             std::log2((double)cfg.rope_theta), st));
  HIP_OK(hipMemcpyAsync(c->at<float>(L.beta), c->at<float>(L.beta_fixed), (size_t)NE * 4,
                        hipMemcpyDeviceToDevice, st));

  LoadArgs la{};
  la.src_k = c->at<uint64_t>(L.src_k);
  la.src_v = c->at<uint64_t>(L.src_v);
  la.items = c->at<int32_t>(L.load_items);
  la.len0 = c->at<int32_t>(L.len0);
  la.page_table = c->at<int32_t>(L.page_table);
  la.kpool = k_pool;
  la.vpool = v_pool;
  la.n_layers = cfg.n_layers;
  la.n_kv_heads = cfg.n_kv_heads;
  la.head_dim = cfg.head_dim;
  la.max_pages = cfg.max_pages;
  la.maxpps = P;
  if (!items.empty()) HIP_OK(launch_load(la, (int)(items.size() / 2), c->bf16, st));
  {
    HostLoader hl(cfg, st);
    for (long s = 0; s < S; ++s) {
      if (!on_host[s]) continue;
      for (int l = 0; l < cfg.n_layers; ++l) {
        r = hl.put(src_k[s], cache_len[s], l, &pt[s * P], false, k_pool);
        if (r == PCED_OK) r = hl.put(src_v[s], cache_len[s], l, &pt[s * P], true, v_pool);
        if (r != PCED_OK) return r;
      }
    }
    r = hl.flush();
    if (r != PCED_OK) return r;
  }

  c->kpool = k_pool;
  c->vpool = v_pool;
  c->dynamic_beta = beta == nullptr;
  c->beta_frozen = false;
  c->t = 0;
  c->loaded = true;
  return PCED_OK;
}

pced_status pced_step(pced_ctx* c, const void* q, const void* k_new, const void* v_new,
                      const void* lm_head, int32_t* tokens_out, const pced_step_out* extra,
                      hipStream_t st) {
  pced_status r = check_ctx(c, true);
  if (r != PCED_OK) return r;
  if (!q || !k_new || !v_new || !lm_head || !tokens_out) return fail(PCED_ERR_INVALID_ARG, "NULL argument");
  // the kernels read q, k_new and v_new in 16-byte units
  if (((uintptr_t)q | (uintptr_t)k_new | (uintptr_t)v_new) % 16)
    return fail(PCED_ERR_INVALID_ARG, "q, k_new and v_new must be 16-byte aligned");
  return run_step(c, q, k_new, v_new, lm_head, tokens_out, 1, extra, st);
}

pced_status pced_generate(pced_ctx* c, int32_t n_steps, const pced_synth* synth, const void* lm_head,
                          int32_t* tokens_out, const pced_step_out* last_extra, hipStream_t st) {
  pced_status r = check_ctx(c, true);
  if (r != PCED_OK) return r;
  if (!synth || !lm_head || !tokens_out) return fail(PCED_ERR_INVALID_ARG, "NULL argument");
  if (n_steps < 1) return fail(PCED_ERR_INVALID_ARG, "n_steps < 1");
  if (synth->first_token < 0 || synth->first_token >= c->cfg.vocab)
    return fail(PCED_ERR_INVALID_ARG, "first_token out of range");
  const int P = c->cfg.max_pages_per_seq;
  for (int s = 0; s < c->S; ++s) {
    const long last = (long)c->len[s] + n_steps - 1;
    const long pidx = last / kPage;
    if (pidx >= P) return fail(PCED_ERR_CAPACITY, "sequence %d cannot hold %d more tokens", s, n_steps);
    for (long p = c->len[s] / kPage; p <= pidx; ++p)
      if (c->page_table[(size_t)s * P + p] < 0)
        return fail(PCED_ERR_CAPACITY, "sequence %d cannot hold %d more tokens", s, n_steps);
  }
  const pced_config& cfg = c->cfg;
  SynthArgs sa{};
  sa.q = c->at<void>(c->lay.syn_q);
  sa.k_new = c->at<void>(c->lay.syn_k);
  sa.v_new = c->at<void>(c->lay.syn_v);
  sa.seq_query = c->at<int32_t>(c->lay.seq_query);
  sa.prev_tok = c->at<int32_t>(c->lay.prev_tok);
  sa.seed = synth->seed;
  sa.value_scale = (float)(std::sqrt(3.0) / 65536.0);
  sa.n_layers = cfg.n_layers;
  sa.qdim = cfg.n_q_heads * cfg.head_dim;
  sa.kvdim = cfg.n_kv_heads * cfg.head_dim;
  sa.first_token = synth->first_token;
  sa.bf16 = c->bf16;
  const double es = (double)esize_of(cfg);
  for (int i = 0; i < n_steps; ++i) {
    sa.t = c->t;
    sa.use_first = c->t == 0;
    {
      ProfScope ps(c, PCED_PROF_SYNTH, (double)c->S * cfg.n_layers * (sa.qdim + 2.0 * sa.kvdim) * es, 0);
      HIP_OK(launch_synth(sa, c->S, st, ps.timing()));
    }
    r = run_step(c, sa.q, sa.k_new, sa.v_new, lm_head, tokens_out + i, n_steps,
                 i == n_steps - 1 ? last_extra : nullptr, st);
    if (r != PCED_OK) return r;
  }
  return PCED_OK;
}

size_t pced_model_bytes(const pced_config* cfg) {
  if (!cfg_valid(cfg, nullptr) || cfg->ffn_dim <= 0) return 0;
  return model_layout(*cfg).total;
}

pced_status pced_pack_model_layer(const pced_config* cfg, int32_t layer, const void* const* tensors, void* model,
                                  hipStream_t st) {
  std::string why;
  if (!cfg_valid(cfg, &why)) return fail(PCED_ERR_INVALID_ARG, "invalid config: %s", why.c_str());
  if (cfg->ffn_dim <= 0) return fail(PCED_ERR_INVALID_ARG, "no decoder stack configured (ffn_dim == 0)");
  if (layer < 0 || layer >= cfg->n_layers) return fail(PCED_ERR_INVALID_ARG, "layer %d out of range", layer);
  if (!tensors || !model) return fail(PCED_ERR_INVALID_ARG, "NULL argument");
  for (int i = 0; i < 9; ++i)
    if (!tensors[i]) return fail(PCED_ERR_INVALID_ARG, "tensor %d is NULL", i);
  const ModelLayout ml = model_layout(*cfg);
  char* lw = (char*)model + (size_t)layer * ml.layer_bytes;
  const int H = cfg->hidden, F = cfg->ffn_dim;
  const int qd = cfg->n_q_heads * cfg->head_dim, kd = cfg->n_kv_heads * cfg->head_dim;
  HIP_OK(hipMemcpyAsync(lw + ml.attn_norm, tensors[0], (size_t)H * 2, hipMemcpyDeviceToDevice, st));
  HIP_OK(hipMemcpyAsync(lw + ml.mlp_norm, tensors[5], (size_t)H * 2, hipMemcpyDeviceToDevice, st));
  // QKV: q tiles, then k tiles, then v tiles (all row counts are multiples of 16)
  const int qkv_tiles = (qd + 2 * kd) / 16;
  HIP_OK(launch_pack_tiles(tensors[1], lw + ml.qkv, qd, H, 1, 0, qkv_tiles, st));
  HIP_OK(launch_pack_tiles(tensors[2], lw + ml.qkv, kd, H, 1, qd / 16, qkv_tiles, st));
  HIP_OK(launch_pack_tiles(tensors[3], lw + ml.qkv, kd, H, 1, (qd + kd) / 16, qkv_tiles, st));
  HIP_OK(launch_pack_tiles(tensors[4], lw + ml.o, H, qd, 1, 0, H / 16, st));
  // gate and up tiles alternate, so a block owning tiles 2j, 2j+1 has both halves of 16 MLP columns
  HIP_OK(launch_pack_tiles(tensors[6], lw + ml.gu, F, H, 2, 0, 2 * F / 16, st));
  HIP_OK(launch_pack_tiles(tensors[7], lw + ml.gu, F, H, 2, 1, 2 * F / 16, st));
  HIP_OK(launch_pack_tiles(tensors[8], lw + ml.down, H, F, 1, 0, H / 16, st));
  // row-major copies: q, k, v rows in order; gate and up 16-row blocks alternating
  const size_t row = (size_t)H * 2;
  HIP_OK(hipMemcpyAsync(lw + ml.qkv_rm, tensors[1], qd * row, hipMemcpyDeviceToDevice, st));
  HIP_OK(hipMemcpyAsync(lw + ml.qkv_rm + qd * row, tensors[2], kd * row, hipMemcpyDeviceToDevice, st));
  HIP_OK(hipMemcpyAsync(lw + ml.qkv_rm + (qd + kd) * row, tensors[3], kd * row, hipMemcpyDeviceToDevice, st));
  HIP_OK(hipMemcpyAsync(lw + ml.o_rm, tensors[4], (size_t)H * qd * 2, hipMemcpyDeviceToDevice, st));
  for (int h = 0; h < 2; ++h)
    HIP_OK(hipMemcpy2DAsync(lw + ml.gu_rm + h * 16 * row, 32 * row, tensors[6 + h], 16 * row, 16 * row, F / 16,
                            hipMemcpyDeviceToDevice, st));
  HIP_OK(hipMemcpyAsync(lw + ml.down_rm, tensors[8], (size_t)H * F * 2, hipMemcpyDeviceToDevice, st));
  return PCED_OK;
}

pced_status pced_pack_model_globals(const pced_config* cfg, const void* embed, const void* final_norm, void* model,
                                    hipStream_t st) {
  std::string why;
  if (!cfg_valid(cfg, &why)) return fail(PCED_ERR_INVALID_ARG, "invalid config: %s", why.c_str());
  if (cfg->ffn_dim <= 0) return fail(PCED_ERR_INVALID_ARG, "no decoder stack configured (ffn_dim == 0)");
  if (!embed || !final_norm || !model) return fail(PCED_ERR_INVALID_ARG, "NULL argument");
  const ModelLayout ml = model_layout(*cfg);
  HIP_OK(hipMemcpyAsync((char*)model + ml.embed, embed, (size_t)cfg->vocab * cfg->hidden * 2,
                        hipMemcpyDeviceToDevice, st));
  HIP_OK(hipMemcpyAsync((char*)model + ml.final_norm, final_norm, (size_t)cfg->hidden * 2,
                        hipMemcpyDeviceToDevice, st));
  return PCED_OK;
}

pced_status pced_model_prefill(pced_ctx* c, const void* model, int32_t n_tokens, const int32_t* tokens,
                               hipStream_t st) {
  pced_status r = check_model(c, model);
  if (r != PCED_OK) return r;
  if (!tokens) return fail(PCED_ERR_INVALID_ARG, "tokens is NULL");
  if (n_tokens < 0) return fail(PCED_ERR_INVALID_ARG, "n_tokens < 0");
  r = check_room(c, n_tokens);
  if (r != PCED_OK) return r;
  // chunks of T suffix tokens: S*T rows per pass through the stack
  const int T = std::max(1, c->lay.pf_rows / c->S);
  for (int i0 = 0; i0 < n_tokens; i0 += T) {
    const int n = std::min(T, n_tokens - i0);
    r = run_prefill_chunk(c, (const char*)model, tokens, n_tokens, i0, n, st);
    if (r != PCED_OK) return r;
    for (int s = 0; s < c->S; ++s) c->len[s] += n;
    c->t += n;
  }
  return PCED_OK;
}

pced_status pced_model_step(pced_ctx* c, const void* model, const void* lm_head, const int32_t* in_tokens,
                            int32_t* tokens_out, const pced_step_out* extra, hipStream_t st) {
  pced_status r = check_model(c, model);
  if (r != PCED_OK) return r;
  if (!lm_head || !in_tokens || !tokens_out) return fail(PCED_ERR_INVALID_ARG, "NULL argument");
  return run_model_step(c, model, lm_head, in_tokens, tokens_out, 1, extra, st);
}

pced_status pced_model_generate(pced_ctx* c, const void* model, const void* lm_head, int32_t n_steps,
                                const int32_t* first_tokens, int32_t* tokens_out, const pced_step_out* last_extra,
                                hipStream_t st) {
  pced_status r = check_model(c, model);
  if (r != PCED_OK) return r;
  if (!lm_head || !first_tokens || !tokens_out) return fail(PCED_ERR_INVALID_ARG, "NULL argument");
  if (n_steps < 1) return fail(PCED_ERR_INVALID_ARG, "n_steps < 1");
  r = check_room(c, n_steps);
  if (r != PCED_OK) return r;
  // step i > 0 feeds the token step i-1 chose, which the fuse also leaves in prev_tok
  const int32_t* prev = c->at<int32_t>(c->lay.prev_tok);
  for (int i = 0; i < n_steps; ++i) {
    r = run_model_step(c, model, lm_head, i == 0 ? first_tokens : prev, tokens_out + i, n_steps,
                       i == n_steps - 1 ? last_extra : nullptr, st);
    if (r != PCED_OK) return r;
  }
  return PCED_OK;
}

pced_status pced_lmhead(pced_ctx* c, const void* x, int32_t n_rows, const void* lm_head, float* logits,
                        hipStream_t st) {
  pced_status r = check_ctx(c, false);
  if (r != PCED_OK) return r;
  if (!x || !lm_head || !logits) return fail(PCED_ERR_INVALID_ARG, "NULL argument");
  if (n_rows < 1 || n_rows > c->cfg.max_seqs)
    return fail(PCED_ERR_INVALID_ARG, "n_rows %d not in [1, %d]", n_rows, c->cfg.max_seqs);
  // the kernel reads whole 48-row tiles of x: stage the rows in the padded buffer
  void* xw = c->at<void>(c->lay.x);
  HIP_OK(launch_copy_rows(x, xw, (size_t)n_rows * c->cfg.hidden * esize_of(c->cfg), st));
  return run_lmhead(c, xw, n_rows, lm_head, logits, st);
}

pced_status pced_lmhead_noalloc(const pced_config* cfg, const void* x, int32_t n_rows, const void* lm_head,
                                float* logits, hipStream_t st) {
  std::string why;
  if (!cfg_valid(cfg, &why)) return fail(PCED_ERR_INVALID_ARG, "invalid config: %s", why.c_str());
  if (!x || !lm_head || !logits) return fail(PCED_ERR_INVALID_ARG, "NULL argument");
  if (n_rows < 1) return fail(PCED_ERR_INVALID_ARG, "n_rows %d < 1", n_rows);
  const size_t row_bytes = (size_t)cfg->hidden * esize_of(*cfg);
  const int wide = cfg->dtype == PCED_BF16 ? lmhead_wide_tiles(n_rows, cfg->vocab, cfg->hidden) : 0;
  LmArgs a{};
  a.w = lm_head;
  a.logits = logits;
  a.M = n_rows;
  a.V = cfg->vocab;
  a.K = cfg->hidden;
  a.rms = cfg->norm == PCED_NORM_RMS;
  if (wide) {
    // the many-row kernel reads only rows < n_rows of x (through its packed
    // copy, which holds the padding): scratch = packed x, then the row scales
    const size_t packed = (size_t)wide * 32 * row_bytes;
    if (packed + (size_t)n_rows * 4 > kNoAllocScratchBytes)
      return fail(PCED_ERR_CAPACITY, "%d rows need %zu bytes of scratch > the %zu available", n_rows,
                  packed + (size_t)n_rows * 4, kNoAllocScratchBytes);
    void* scratch = nullptr;
    HIP_OK(noalloc_scratch(&scratch));
    a.x = x;
    a.x_packed = scratch;
    a.rho_buf = (float*)((char*)scratch + packed);
  } else {
    // the other kernels read whole 16-row tiles of x: stage the rows, padded with zero rows
    const size_t rows = (size_t)ceil_div(n_rows, 16) * 16;
    if (rows * row_bytes > kNoAllocScratchBytes)
      return fail(PCED_ERR_CAPACITY, "%d rows of %zu bytes need %zu bytes of scratch > the %zu available", n_rows,
                  row_bytes, rows * row_bytes, kNoAllocScratchBytes);
    void* scratch = nullptr;
    HIP_OK(noalloc_scratch(&scratch));
    char* xs = (char*)scratch;
    HIP_OK(launch_copy_rows(x, xs, (size_t)n_rows * row_bytes, st));
    HIP_OK(launch_zero_bytes(xs + (size_t)n_rows * row_bytes, (rows - n_rows) * row_bytes, st));
    a.x = xs;
  }
  HIP_OK(launch_lmhead(a, cfg->dtype == PCED_BF16, st));
  return PCED_OK;
}

pced_status pced_fuse(pced_ctx* c, const float* logits, int32_t refresh_beta, int32_t* tokens_out,
                      const pced_step_out* extra, hipStream_t st) {
  pced_status r = check_ctx(c, true);
  if (r != PCED_OK) return r;
  if (!logits || !tokens_out) return fail(PCED_ERR_INVALID_ARG, "NULL argument");
  if (c->dynamic_beta && !refresh_beta && !c->beta_frozen)
    return fail(PCED_ERR_STATE, "dynamic beta has not been computed yet (pass refresh_beta)");
  return run_fuse(c, logits, refresh_beta != 0, tokens_out, 1, extra, st);
}

pced_status pced_stream_read(const void* src, size_t bytes, uint32_t* xor_out, hipStream_t st) {
  if (!xor_out || (!src && bytes > 0)) return fail(PCED_ERR_INVALID_ARG, "NULL argument");
  if ((uintptr_t)src % 16 != 0 || bytes % 16 != 0)
    return fail(PCED_ERR_INVALID_ARG, "src must be 16-byte aligned and bytes a multiple of 16 (bytes = %zu)", bytes);
  if ((uintptr_t)xor_out % 4 != 0) return fail(PCED_ERR_INVALID_ARG, "xor_out is not 4-byte aligned");
  if (!is_device_memory(xor_out) || (bytes > 0 && !is_device_memory(src)))
    return fail(PCED_ERR_INVALID_ARG, "src and xor_out must be device memory");
  int dev = 0, cus = 0;
  HIP_OK(hipGetDevice(&dev));
  HIP_OK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  if (bytes == 0) {
    HIP_OK(launch_stream_read(nullptr, 0, xor_out, cus, st));
    return PCED_OK;
  }
  hipDeviceptr_t base = nullptr;
  size_t size = 0;
  if (hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)src) != hipSuccess) {
    (void)hipGetLastError();
    return fail(PCED_ERR_INVALID_ARG, "src is not inside a device allocation");
  }
  if ((const char*)src + bytes > (const char*)base + size)
    return fail(PCED_ERR_INVALID_ARG, "%zu bytes from src run past the end of its allocation", bytes);
  HIP_OK(launch_stream_read(src, bytes, xor_out, cus, st));
  return PCED_OK;
}

pced_status pced_relevance(int32_t mode, int32_t n, const float* retrieval, const float* reranker_logits,
                           float* relevance) {
  if (!retrieval || !relevance) return fail(PCED_ERR_INVALID_ARG, "NULL argument");
  if (n < 0) return fail(PCED_ERR_INVALID_ARG, "n = %d", n);
  if (mode != PCED_SCORE_DENSE && mode != PCED_SCORE_COLBERT && mode != PCED_SCORE_SPARSE)
    return fail(PCED_ERR_INVALID_ARG, "unknown score mode %d", mode);
  for (int32_t k = 0; k < n; ++k)
    if (std::isnan(retrieval[k]) || (reranker_logits && std::isnan(reranker_logits[k])))
      return fail(PCED_ERR_INVALID_ARG, "score %d is NaN", k);
  const double eps = 1e-8, top = 1.0 - eps;
  auto clip = [&](double x) { return std::min(std::max(x, 0.0), top); };
  for (int32_t k = 0; k < n; ++k) {
    const double s = retrieval[k];
    const double r_ret = mode == PCED_SCORE_SPARSE ? clip(2.0 / M_PI * std::atan(std::max(s, 0.0)))
                                                   : clip((s + 1.0) / 2.0);
    double r = r_ret;
    if (reranker_logits) {
      const double r_rer = clip(1.0 / (1.0 + std::exp(-(double)reranker_logits[k])));
      r = 2.0 * r_ret * r_rer / (r_ret + r_rer + eps);
    }
    relevance[k] = (float)r;
  }
  return PCED_OK;
}

pced_status pced_read_cache(pced_ctx* c, int32_t seq, int32_t layer, int32_t start, int32_t count, void* k_out,
                            void* v_out, hipStream_t st) {
  pced_status r = check_ctx(c, true);
  if (r != PCED_OK) return r;
  if (!k_out || !v_out) return fail(PCED_ERR_INVALID_ARG, "NULL argument");
  if (seq < 0 || seq >= c->S) return fail(PCED_ERR_INVALID_ARG, "seq %d not in [0, %d)", seq, c->S);
  if (layer < 0 || layer >= c->cfg.n_layers)
    return fail(PCED_ERR_INVALID_ARG, "layer %d not in [0, %d)", layer, c->cfg.n_layers);
  if (start < 0 || count < 0 || (long)start + count > c->len[seq])
    return fail(PCED_ERR_INVALID_ARG, "tokens [%d, %ld) beyond the %d of sequence %d", start, (long)start + count,
                c->len[seq], seq);
  if (count == 0) return PCED_OK;
  ReadCacheArgs a{};
  a.kpool = c->kpool;
  a.vpool = c->vpool;
  a.page_table = c->at<int32_t>(c->lay.page_table);
  a.k_out = k_out;
  a.v_out = v_out;
  a.seq = seq;
  a.layer = layer;
  a.start = start;
  a.count = count;
  a.n_kv_heads = c->cfg.n_kv_heads;
  a.head_dim = c->cfg.head_dim;
  a.max_pages = c->cfg.max_pages;
  a.maxpps = c->cfg.max_pages_per_seq;
  a.bf16 = c->bf16;
  HIP_OK(launch_read_cache(a, st));
  return PCED_OK;
}

pced_status pced_get_lengths(const pced_ctx* c, int32_t* out, int32_t capacity) {
  pced_status r = check_ctx(c, true);
  if (r != PCED_OK) return r;
  if (!out || capacity < c->S) return fail(PCED_ERR_INVALID_ARG, "output too small");
  std::copy(c->len.begin(), c->len.end(), out);
  return PCED_OK;
}

pced_status pced_profile_enable(pced_ctx* c, int32_t on) {
  pced_status r = check_ctx(c, false);
  if (r != PCED_OK) return r;
  if (on) {
    for (auto& rec : c->recs) { c->ev_free.push_back(rec.a); c->ev_free.push_back(rec.b); }
    c->recs.clear();
    c->totals = pced_profile{};
  }
  c->prof = on != 0;
  return PCED_OK;
}

pced_status pced_profile_read(pced_ctx* c, pced_profile* out) {
  pced_status r = check_ctx(c, false);
  if (r != PCED_OK) return r;
  if (!out) return fail(PCED_ERR_INVALID_ARG, "out is NULL");
  for (auto& rec : c->recs) {
    float ms = 0.f;
    HIP_OK(hipEventElapsedTime(&ms, rec.a, rec.b));
    c->totals.launches[rec.cls] += 1;
    c->totals.total_ms[rec.cls] += ms;
    c->totals.bytes[rec.cls] += rec.bytes;
    c->totals.flops[rec.cls] += rec.flops;
    c->ev_free.push_back(rec.a);
    c->ev_free.push_back(rec.b);
  }
  c->recs.clear();
  *out = c->totals;
  return PCED_OK;
}

}  // extern "C"
