// gfx950 kernels of the PCED decode step (Parallel Context-of-Experts Decoding,
// arXiv 2601.08670, Section 3).
//
// KV pool tile layout. A tile is one (layer, page, kv-head): 16 tokens x D.
//   bf16 K tile: element (t, d) at ((d/32)*64 + t + 16*((d%32)/8))*8 + d%8.
//     Lane l's 16-byte load number i is exactly the A operand of
//     v_mfma_f32_16x16x32_bf16 for the 16x32 block (tokens, dims 32i..32i+31):
//     row t = l%16, k = 8*(l/16)..+7.
//   bf16 V tile: element (t, d) at ((j/2*64 + d%16 + 16*(t/4))*2 + j%2)*4 + t%4,
//     j = d/16. Lane l's 16-byte load number jj holds the A operands of two
//     v_mfma_f32_16x16x16_bf16 for V^T blocks j = 2jj, 2jj+1: row d = 16j + l%16,
//     k = tokens 4*(l/16)..+3.
//   f32 tiles are row-major [t][d].
// Every wave load of a page is therefore a contiguous 1 KiB.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>
#include <utility>

#include "pced_internal.h"

namespace pced {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kNegInf = -INFINITY;

__device__ __forceinline__ float bf2f(uint32_t b) { return __uint_as_float(b << 16); }

// round-to-nearest-even float -> bf16 bits (finite inputs)
__device__ __forceinline__ uint32_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }


typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// 16-byte load of data a launch reads once (KV pages, LM-head and projection
// weights in a decode step): with STREAM it carries the non-temporal hint and
// streams through the caches without displacing what is reused (partial
// states, outputs, q and x rows). Launches that read the same bytes several
// times (the prefill's row groups and virtual rows, the LM head's row groups)
// use plain loads, so that the repeats hit the caches.
template <bool STREAM>
__device__ __forceinline__ uint4 ld_w(const uint4* p) {
  if constexpr (STREAM) {
    const u32x4 v = __builtin_nontemporal_load((const u32x4*)p);
    return make_uint4(v.x, v.y, v.z, v.w);
  } else {
    return *p;
  }
}

// ------------------------------------------------------------------ utilities

__global__ void k_fill_i32(int32_t* p, int32_t v, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = v;
}

__global__ void k_zero_u32(uint32_t* p, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

// ------------------------------------------------------------- cache loading

// One block per (sequence, logical page) item and layer: copies the page's
// tokens of every kv-head from the contiguous [L][len][Hkv][D] source into the
// pool tiles, zero-filling slots past the sequence's length.
template <bool BF16>
__global__ __launch_bounds__(256) void k_load(LoadArgs a) {
  const int item = blockIdx.x, l = blockIdx.y;
  const int s = a.items[2 * item], p = a.items[2 * item + 1];
  const int len = a.len0[s];
  const int phys = a.page_table[(size_t)s * a.maxpps + p];
  const int Hkv = a.n_kv_heads, D = a.head_dim;
  const size_t tile = (size_t)kPage * D;
  const size_t tile0 = ((size_t)l * a.max_pages + phys) * Hkv;
  const int n = Hkv * kPage * D;
  for (int idx = threadIdx.x; idx < n; idx += blockDim.x) {
    const int g = idx / (kPage * D), rem = idx % (kPage * D);
    const int t = rem / D, d = rem % D;
    const int tok = p * kPage + t;
    const size_t src = (((size_t)l * len + tok) * Hkv + g) * D + d;
    const size_t base = (tile0 + g) * tile;
    if (BF16) {
      const uint16_t* sk = (const uint16_t*)a.src_k[s];
      const uint16_t* sv = (const uint16_t*)a.src_v[s];
      const uint16_t kv = tok < len ? sk[src] : 0, vv = tok < len ? sv[src] : 0;
      ((uint16_t*)a.kpool)[base + kswz(t, d)] = kv;
      ((uint16_t*)a.vpool)[base + vswz(t, d)] = vv;
    } else {
      const float* sk = (const float*)a.src_k[s];
      const float* sv = (const float*)a.src_v[s];
      ((float*)a.kpool)[base + (size_t)t * D + d] = tok < len ? sk[src] : 0.f;
      ((float*)a.vpool)[base + (size_t)t * D + d] = tok < len ? sv[src] : 0.f;
    }
  }
}

// --------------------------------------------- shared-history append + plan

// Balanced attention plan. The pages of all sequences (after this step's
// append), concatenated in sequence order, are cut into C chunks: chunk c holds
// global pages [chunk_lo(c), chunk_lo(c + 1)) with chunk_lo(c) = floor(c P / C),
// so chunk sizes differ by at most one page and every wave of the attention
// launch streams the same amount of cache.
__device__ __forceinline__ long chunk_lo(long c, long P, long C) { return c * P / C; }
// the chunk holding global page u: the largest c with chunk_lo(c) <= u
__device__ __forceinline__ int chunk_of(long u, long P, long C) { return (int)(((u + 1) * C - 1) / P); }

// Blocks 0 .. S*L-1 (when k_new is given): write step t's K/V row of (sequence, layer) into slot
// len0 + t of the sequence's pages (Section 3: the chosen token joins every
// expert's history). Block S*L + s plans sequence s for this step's length
// len0 + t + 1: the chunks it meets, its segment descriptor in each (the
// sequence's position among the chunk's segments comes from walking back over
// the sequences that reach into the chunk), and the physical id of each of its
// pages at the page's place in its chunk.
template <bool BF16>
__global__ __launch_bounds__(128) void k_append(AppendArgs a) {
  const int S = a.n_seqs, L = a.n_layers;
  const int n_app = a.k_new ? S * L : 0;  // without K/V rows (written elsewhere) only the planning blocks run
  if ((int)blockIdx.x >= n_app) {
    const int s = blockIdx.x - n_app;
    const long P = a.total_pages, C = a.n_chunks;
    auto pages_of = [&](int r) { return max(a.min_pages, (a.len0[r] + a.t + 1 + kPage - 1) / kPage); };
    // first global page of this sequence: sum over earlier sequences; the page
    // counts of the kMaxSeg sequences just before s also go to LDS for the walk
    // back below (one round of loads instead of a chain of dependent ones)
    __shared__ int red[2];
    __shared__ int back[kMaxSeg];
    __shared__ int k_first;
    int part = 0;
    for (int r = threadIdx.x; r < s; r += blockDim.x) {
      const int p = pages_of(r);
      part += p;
      if (r >= s - kMaxSeg) back[r - (s - kMaxSeg)] = p;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) part += __shfl_xor(part, o);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = part;
    const int len = a.len0[s] + a.t + 1;
    const int ps_own = (len + kPage - 1) / kPage, ps = max(a.min_pages, ps_own);
    __syncthreads();
    const long pre = red[0] + red[1];
    const int c0 = chunk_of(pre, P, C), c1 = chunk_of(pre + ps - 1, P, C);
    if (threadIdx.x == 0) {
      a.nparts[s] = c1 - c0 + 1;
      // segments of chunk c0 before this one: earlier sequences ending after its start
      const long b0 = chunk_lo(c0, P, C);
      long end = pre;
      int k = 0;
      for (int r = s - 1; r >= 0 && end > b0 && k < kMaxSeg; --r) {  // r >= s - kMaxSeg
        ++k;
        end -= back[r - (s - kMaxSeg)];
      }
      k_first = k;
    }
    __syncthreads();
    for (int c = c0 + (int)threadIdx.x; c <= c1; c += blockDim.x) {
      const long lo_c = chunk_lo(c, P, C), hi_c = chunk_lo(c + 1, P, C);
      const long lo = max(pre, lo_c), hi = min(pre + ps, hi_c);
      const int k = c == c0 ? k_first : 0;
      const int i0 = (int)(lo - lo_c), pa = (int)(lo - pre);
      if (k < kMaxSeg) {
        a.seg[((size_t)c * kMaxSeg + k) * 2] = make_int4(s, i0, pa - i0, min(len, (int)(hi - pre) * kPage));
        a.seg[((size_t)c * kMaxSeg + k) * 2 + 1] = make_int4(c - c0, c1 - c0 + 1, len, 0);
      }
      if (hi == hi_c) a.chunk_info[c] = make_int2(k + 1, (int)(hi_c - lo_c));  // last segment of chunk c
    }
    const int32_t* pt = a.page_table + (size_t)s * a.maxpps;
    for (int p = threadIdx.x; p < ps; p += blockDim.x) {
      const long u = pre + p;
      const int c = chunk_of(u, P, C);
      a.work_pages[(size_t)c * kMaxSplitPages + (u - chunk_lo(c, P, C))] = pt[min(p, ps_own - 1)];
    }
    return;
  }
  const int s = blockIdx.x / L, l = blockIdx.x % L;
  const int pos = a.len0[s] + a.t;
  const int phys = a.page_table[(size_t)s * a.maxpps + pos / kPage];
  const int slot = pos % kPage;
  const int Hkv = a.n_kv_heads, D = a.head_dim;
  const size_t tile = (size_t)kPage * D;
  const size_t tile0 = ((size_t)l * a.max_pages + phys) * Hkv;
  const size_t src0 = ((size_t)s * L + l) * Hkv * D;
  if constexpr (BF16) {
    // Only whole 32-byte sectors are written: a store that fills part of a
    // sector leaves a partly valid line behind, and merging it with memory
    // later slows the attention launches that read the page. The sector is
    // read back and only this slot's bytes change, so the neighbouring slots
    // keep what they hold.
    // The stores carry the non-temporal hint: the rows go out to memory during
    // this launch instead of staying dirty in the caches, where the next
    // attention launches, streaming every page of the layer, would pay for
    // their write-back. D is 64 or 128.
    const uint16_t* kn = (const uint16_t*)a.k_new + src0;
    const uint16_t* vn = (const uint16_t*)a.v_new + src0;
    // K: 8 dims of one token are 16 contiguous bytes, and a sector holds them
    // for the token pair (slot & ~1, slot | 1)
    const bool odd = slot & 1;
    for (int i0 = 8 * threadIdx.x; i0 < Hkv * D; i0 += 8 * blockDim.x) {
      const int g = i0 / D, d0 = i0 % D;
      uint4* sec = (uint4*)((uint16_t*)a.kpool + (tile0 + g) * tile + kswz(slot & ~1, d0));
      const uint4 kv = *(const uint4*)(kn + i0);
      const uint4 other = sec[odd ? 0 : 1];
      const uint4 lo = odd ? other : kv, hi = odd ? kv : other;
      __builtin_nontemporal_store(u32x4{lo.x, lo.y, lo.z, lo.w}, (u32x4*)sec);
      __builtin_nontemporal_store(u32x4{hi.x, hi.y, hi.z, hi.w}, (u32x4*)sec + 1);
    }
    // V: the 4 tokens of a slot group share each 8-byte unit of one dim, and
    // the 16 units of dims d0 .. d0+7 and d0+16 .. d0+23 (d0 = 32 jj + 8 h)
    // are 128 contiguous bytes: unit 2 i holds dim d0 + i, unit 2 i + 1 dim
    // d0 + 16 + i. A thread owns one such run.
    const int q4 = slot & 3, sh = 16 * (q4 & 1);
    for (int v = threadIdx.x; v < Hkv * D / 16; v += blockDim.x) {
      const int g = v / (D / 16), r = v % (D / 16);
      const int d0 = 32 * (r >> 1) + 8 * (r & 1);
      uint4* run = (uint4*)((uint16_t*)a.vpool + (tile0 + g) * tile + vswz(slot & ~3, d0));
      const uint4 va = *(const uint4*)(vn + g * D + d0), vb = *(const uint4*)(vn + g * D + d0 + 16);
      uint4 cur[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) cur[k] = run[k];
      const uint32_t wa[4] = {va.x, va.y, va.z, va.w}, wb[4] = {vb.x, vb.y, vb.z, vb.w};
      auto put = [&](uint32_t& w, uint32_t e) { w = (w & ~(0xFFFFu << sh)) | ((e & 0xFFFFu) << sh); };
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const uint32_t e0 = wa[k >> 1] >> (16 * (k & 1)), e1 = wb[k >> 1] >> (16 * (k & 1));
        if (q4 < 2) { put(cur[k].x, e0); put(cur[k].z, e1); }
        else { put(cur[k].y, e0); put(cur[k].w, e1); }
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) __builtin_nontemporal_store(u32x4{cur[k].x, cur[k].y, cur[k].z, cur[k].w}, (u32x4*)run + k);
    }
  } else {
    // row-major fp32 tiles: a token's row is whole lines
    for (int i0 = 4 * threadIdx.x; i0 < Hkv * D; i0 += 4 * blockDim.x) {
      const size_t base = (tile0 + i0 / D) * tile + (size_t)slot * D + i0 % D;
      const float4 kv = *(const float4*)((const float*)a.k_new + src0 + i0);
      const float4 vv = *(const float4*)((const float*)a.v_new + src0 + i0);
      *(float4*)((float*)a.kpool + base) = kv;
      *(float4*)((float*)a.vpool + base) = vv;
    }
  }
}

// ----------------------------------------------------------- decode attention

// Prefill token groups (a.tq tokens per plan item): item v is token group
// v % ng of sequence v / ng (ng = ceil(tq_T / tq)); of its a.group columns per
// kv-head g, column c is token c / gk of the group and q-head g gk + c % gk
// (gk = a.group / tq). Returns the physical row (s tq_T + token) and q-head,
// the token clamped to the group's last, and whether the token exists.
struct MqCol {
  int row, head, valid;
};
__device__ __forceinline__ MqCol mq_col(const AttnArgs& a, int v, int g, int c) {
  const int gk = a.group / a.tq, ng = (a.tq_T + a.tq - 1) / a.tq;
  const int s = v / ng, j = v - s * ng;
  const int last = min(a.tq, a.tq_T - a.tq * j) - 1;
  const int u = c / gk;
  return MqCol{s * a.tq_T + a.tq * j + min(u, last), g * gk + c % gk, u <= last};
}
// Tokens between column c's own token and the last token of group v: the
// column's keys end that many positions before the group's.
__device__ __forceinline__ int mq_end_off(const AttnArgs& a, int v, int c) {
  const int gk = a.group / a.tq, ng = (a.tq_T + a.tq - 1) / a.tq;
  const int j = v % ng;
  const int last = min(a.tq, a.tq_T - a.tq * j) - 1;
  return last - min(c / gk, last);
}

// Write 4 consecutive output dims of one q-head: fp32 debug copy, the layer
// output in the storage type, and (last layer) the fp32 value of the stored x.
// MQ: s is a prefill token group and head = kv-head x group + column (mq_col);
// columns of tokens past the group's end are not written.
template <bool BF16, bool MQ = false>
__device__ __forceinline__ void write_o4(const AttnArgs& a, int s, int head, int d, int D, float4 o) {
  const int Hq = a.n_q_heads;
  if constexpr (MQ) {
    const MqCol m = mq_col(a, s, head / a.group, head % a.group);
    if (!m.valid) return;
    s = m.row;
    head = m.head;
  }
  const size_t xo = (size_t)s * Hq * D + (size_t)head * D + d;
  if (a.attn_out) {
    float4* p = (float4*)(a.attn_out + (((size_t)s * a.n_layers + a.layer) * Hq + head) * D + d);
    *p = o;
  }
  if (BF16) {
    const uint32_t b0 = f2bf(o.x), b1 = f2bf(o.y), b2 = f2bf(o.z), b3 = f2bf(o.w);
    uint2 pk;
    pk.x = b0 | (b1 << 16);
    pk.y = b2 | (b3 << 16);
    *(uint2*)((uint16_t*)a.x_out + xo) = pk;
    if (a.is_last_layer && a.hidden_out)
      *(float4*)(a.hidden_out + xo) = make_float4(bf2f(b0), bf2f(b1), bf2f(b2), bf2f(b3));
  } else {
    *(float4*)((float*)a.x_out + xo) = o;
    if (a.is_last_layer && a.hidden_out) *(float4*)(a.hidden_out + xo) = o;
  }
}

// Merge of a sequence's split partial states:
//   m* = max_j m_j,  o = sum_j acc_j 2^(m_j - m*) / sum_j l_j 2^(m_j - m*),
// with acc_j = l_j o_j for the bf16 path, whose partials hold the normalised
// output o_j in bf16 (the fp32 path keeps acc_j in fp32). Sequences that fit
// one split were written directly by the attention kernel.
//
// bf16: one wave per item (sequence, kv-head, q-head), in the merge kernel and
// in the prologue of the next layer's attention launch alike, through the
// functions below (same operations in the same order: bit-identical results).
// Splits go in groups of 16, merged online. Within a group, lane l loads 8
// dims (16 bytes) of split 4 i + l / (D/8) in load i (D = 128: 4 splits per
// load), and lane l % 16 holds (m, l) of split l % 16; a lane sums its splits in
// order, then the lane groups are added by a butterfly (every group ends with
// the same bits). Slots past the split count are read but never used.
template <int D>
struct MergeShape {
  static constexpr int LPS = D / 8;     // lanes per split
  static constexpr int SPI = 64 / LPS;  // splits per load
  static constexpr int NI = 16 / SPI;   // loads per group of 16 splits
};

template <int D>
struct MergeRegs {
  uint4 v[MergeShape<D>::NI];
  float2 ml;
};

template <int D>
__device__ __forceinline__ void merge_load(MergeRegs<D>& R, const uint16_t* acc, const float* ml, size_t w0,
                                           int stride, int G, int h, int j0, int lane) {
  using M = MergeShape<D>;
  const int last = stride - 1;
  R.ml = *(const float2*)(ml + ((w0 + min(j0 + (lane & 15), last)) * G + h) * 2);
#pragma unroll
  for (int i = 0; i < M::NI; ++i) {
    const int j = j0 + i * M::SPI + lane / M::LPS;
    R.v[i] = *(const uint4*)(acc + ((w0 + min(j, last)) * G + h) * D + 8 * (lane % M::LPS));
  }
}

template <int D>
__device__ __forceinline__ void merge_group(const MergeRegs<D>& R, int j0, int n, int lane, float& m_run,
                                            float& den, float (&num)[8]) {
#pragma clang fp contract(off)
  using M = MergeShape<D>;
  const bool valid = j0 + (lane & 15) < n;
  const float mj = valid ? R.ml.x : kNegInf;
  float mg = mj;
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) mg = fmaxf(mg, __shfl_xor(mg, o));
  mg = fmaxf(mg, m_run);  // uniform: every 16-lane group holds all 16 splits
  const float wj = valid ? exp2f(mj - mg) : 0.f;
  const float r = exp2f(m_run - mg);
  den *= r;
#pragma unroll
  for (int e = 0; e < 8; ++e) num[e] *= r;
  m_run = mg;
#pragma unroll
  for (int i = 0; i < M::NI; ++i) {
    const int jj = i * M::SPI + lane / M::LPS;
    const float lj = __shfl(R.ml.y, jj), w = __shfl(wj, jj);
    if (j0 + jj < n) {
      const float wv = lj * w;  // weight of the stored (normalised) values
      den = fmaf(lj, w, den);
      const uint32_t b[4] = {R.v[i].x, R.v[i].y, R.v[i].z, R.v[i].w};
#pragma unroll
      for (int e = 0; e < 8; ++e) num[e] = fmaf(bf2f((b[e >> 1] >> (16 * (e & 1))) & 0xFFFFu), wv, num[e]);
    }
  }
}

// Sum over the lane groups and store: x_out (bf16), attn_out at `layer` and,
// for the last layer, hidden_out (fp32 of the stored x).
template <int D>
__device__ __forceinline__ void merge_store(const AttnArgs& a, int s, int head, int layer, bool last_layer,
                                            int lane, float den, float (&num)[8]) {
#pragma clang fp contract(off)
  using M = MergeShape<D>;
#pragma unroll
  for (int o = M::LPS; o < 64; o <<= 1) {
    den += __shfl_xor(den, o);
#pragma unroll
    for (int e = 0; e < 8; ++e) num[e] += __shfl_xor(num[e], o);
  }
  if (lane >= M::LPS) return;
  const float inv = 1.0f / den;
  float o[8];
  uint32_t b[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    o[e] = num[e] * inv;
    b[e] = f2bf(o[e]);
  }
  const int d = 8 * lane;
  const size_t row = (size_t)s * a.n_q_heads + head;
  *(uint4*)((uint16_t*)a.x_out + row * D + d) =
      make_uint4(b[0] | (b[1] << 16), b[2] | (b[3] << 16), b[4] | (b[5] << 16), b[6] | (b[7] << 16));
  if (a.attn_out) {
    float* p = a.attn_out + (((size_t)s * a.n_layers + layer) * a.n_q_heads + head) * D + d;
    *(float4*)p = make_float4(o[0], o[1], o[2], o[3]);
    *(float4*)(p + 4) = make_float4(o[4], o[5], o[6], o[7]);
  }
  if (last_layer && a.hidden_out) {
    float* p = a.hidden_out + row * D + d;
    *(float4*)p = make_float4(bf2f(b[0]), bf2f(b[1]), bf2f(b[2]), bf2f(b[3]));
    *(float4*)(p + 4) = make_float4(bf2f(b[4]), bf2f(b[5]), bf2f(b[6]), bf2f(b[7]));
  }
}

// The whole merge of item `it` whose first group is already in R.
template <int D>
__device__ __forceinline__ void merge_item(const AttnArgs& a, MergeRegs<D>& R, const uint16_t* acc,
                                           const float* ml, int s, int g, int h, int n, int layer,
                                           bool last_layer, int lane) {
  if (n <= 1) return;  // written directly by the attention kernel
  const size_t w0 = (size_t)(s * a.n_kv_heads + g) * a.split_stride;
  float m_run = kNegInf, den = 0.f;
  float num[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int j0 = 0; j0 < n; j0 += 16) {
    if (j0 > 0) merge_load<D>(R, acc, ml, w0, a.split_stride, a.group, h, j0, lane);
    merge_group<D>(R, j0, n, lane, m_run, den, num);
  }
  merge_store<D>(a, s, g * a.group + h, layer, last_layer, lane, den, num);
}

// The merge as a launch of its own: one wave per item.
template <int D>
__global__ __launch_bounds__(64) void k_attn_combine_bf16(AttnArgs a) {
  const int lane = threadIdx.x;
  const int G = a.group, Hkv = a.n_kv_heads;
  const int it = blockIdx.x;
  const int s = it / (Hkv * G), g = (it / G) % Hkv, h = it % G;
  const int n = a.nparts[s];
  const uint16_t* acc = (const uint16_t*)a.part_acc;
  MergeRegs<D> R;
  merge_load<D>(R, acc, a.part_ml, (size_t)(s * Hkv + g) * a.split_stride, a.split_stride, G, h, 0, lane);
  merge_item<D>(a, R, acc, a.part_ml, s, g, h, n, a.layer, a.is_last_layer != 0, lane);
}

// The merge for the prefill's token groups, whose items are many and mostly
// split in a few parts: one wave per (item, kv-head), each lane merging whole
// 8-dim units (column h, dims d .. d+7) over the parts in order, with the same
// formula as above (m* = max_j m_j, weights l_j 2^(m_j - m*) on the stored
// normalised outputs) and no cross-lane traffic. Parts of a column without keys
// hold l = 0 and zeros.
template <int D>
__global__ __launch_bounds__(256) void k_attn_combine_mq(AttnArgs a) {
#pragma clang fp contract(off)
  const int lane = threadIdx.x & 63;
  const int G = a.group, Hkv = a.n_kv_heads;
  const int wv = blockIdx.x * 4 + (int)(threadIdx.x >> 6);
  if (wv >= a.n_seqs * Hkv) return;
  const int s = wv / Hkv, g = wv - s * Hkv;
  const int n = a.nparts[s];
  if (n <= 1) return;  // written directly by the attention kernel
  const size_t w0 = (size_t)wv * a.split_stride;
  const uint16_t* acc = (const uint16_t*)a.part_acc;
  for (int u = lane; u < G * (D / 8); u += 64) {
    const int h = u / (D / 8), d = 8 * (u % (D / 8));
    float mx = kNegInf;
    for (int j = 0; j < n; ++j) mx = fmaxf(mx, a.part_ml[((w0 + j) * G + h) * 2]);
    float den = 0.f, num[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < n; ++j) {
      const float2 ml = *(const float2*)(a.part_ml + ((w0 + j) * G + h) * 2);
      const uint4 v = *(const uint4*)(acc + ((w0 + j) * G + h) * D + d);
      const float wt = ml.y * exp2f(ml.x - mx);
      den += wt;
      const uint32_t b[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) num[e] = fmaf(bf2f((b[e >> 1] >> (16 * (e & 1))) & 0xFFFFu), wt, num[e]);
    }
    const MqCol m = mq_col(a, s, g, h);
    if (!m.valid) continue;
    const float inv = 1.0f / den;
    float o[8];
    uint32_t bb[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      o[e] = num[e] * inv;
      bb[e] = f2bf(o[e]);
    }
    const size_t row = (size_t)m.row * a.n_q_heads + m.head;
    *(uint4*)((uint16_t*)a.x_out + row * D + d) = make_uint4(bb[0] | (bb[1] << 16), bb[2] | (bb[3] << 16),
                                                            bb[4] | (bb[5] << 16), bb[6] | (bb[7] << 16));
    if (a.attn_out) {
      float* p = a.attn_out + (((size_t)m.row * a.n_layers + a.layer) * a.n_q_heads + m.head) * D + d;
      *(float4*)p = make_float4(o[0], o[1], o[2], o[3]);
      *(float4*)(p + 4) = make_float4(o[4], o[5], o[6], o[7]);
    }
    if (a.is_last_layer && a.hidden_out) {
      float* p = a.hidden_out + row * D + d;
      *(float4*)p = make_float4(bf2f(bb[0]), bf2f(bb[1]), bf2f(bb[2]), bf2f(bb[3]));
      *(float4*)(p + 4) = make_float4(bf2f(bb[4]), bf2f(bb[5]), bf2f(bb[6]), bf2f(bb[7]));
    }
  }
}

// fp32: one block per (sequence, kv-head); each thread owns 4 output dims of
// one head and issues the loads of up to 16 splits at once, merging further
// groups of 16 online.
__global__ __launch_bounds__(128) void k_attn_combine_f32(AttnArgs a, int D) {
  constexpr int J = 16;
  const int s = blockIdx.x / a.n_kv_heads, g = blockIdx.x % a.n_kv_heads;
  const int G = a.group, stride = a.split_stride;
  const size_t w0 = (size_t)blockIdx.x * stride;
  const int nsplit = a.nparts[s];
  for (int idx = threadIdx.x; idx < G * D / 4; idx += blockDim.x) {
    const int h = (idx * 4) / D, d = (idx * 4) % D;
    float m_run = kNegInf, den = 0.f;
    float4 num = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int j0 = 0; j0 < max(nsplit, 1); j0 += J) {
      float mj[J], lj[J];
      float4 vj[J];
#pragma unroll
      for (int u = 0; u < J; ++u) {
        const size_t wj = w0 + min(j0 + u, stride - 1);
        mj[u] = a.part_ml[(wj * G + h) * 2];
        lj[u] = a.part_ml[(wj * G + h) * 2 + 1];
        vj[u] = *(const float4*)(a.part_acc + (wj * G + h) * D + d);
      }
      if (nsplit <= 1) return;  // written directly by the attention kernel
      float mg = m_run;
#pragma unroll
      for (int u = 0; u < J; ++u)
        if (j0 + u < nsplit) mg = fmaxf(mg, mj[u]);
      const float r = exp2f(m_run - mg);
      den *= r; num.x *= r; num.y *= r; num.z *= r; num.w *= r;
#pragma unroll
      for (int u = 0; u < J; ++u) {
        if (j0 + u < nsplit) {
          const float w = exp2f(mj[u] - mg);
          den = fmaf(lj[u], w, den);
          num.x = fmaf(vj[u].x, w, num.x); num.y = fmaf(vj[u].y, w, num.y);
          num.z = fmaf(vj[u].z, w, num.z); num.w = fmaf(vj[u].w, w, num.w);
        }
      }
      m_run = mg;
    }
    const float inv = 1.0f / den;
    write_o4<false>(a, s, g * G + h, d, D, make_float4(num.x * inv, num.y * inv, num.z * inv, num.w * inv));
  }
}

// Flash decoding for bf16 caches over the balanced plan, one wave per (chunk,
// kv-head). The G q-heads of the kv-head ride in the N dimension of the matrix
// cores, so every K/V byte is read once for all of them:
//   S^T[16 tok x 16 heads] = K[16 x D] Q^T          (D/32 x 16x16x32 MFMA)
//   O^T[D x 16 heads]     += V^T[D x 16 tok] P^T    (D/16 x 16x16x16 MFMA)
// P comes straight out of the S^T accumulator layout (lane l: head l%16,
// tokens 4*(l/16)..+3), which is the B operand layout of the second product.
// Online softmax in base 2 with log2(e)/sqrt(D) folded into the score scale.
// A chunk may span several sequences. At each segment switch the wave stores
// the finished segment (the final output when the sequence lies in this chunk
// alone, else a partial state for the merge kernel) and continues with the next
// sequence's q, staged in LDS by the prologue, and a fresh softmax state; the
// page stream itself does not stop at a switch.
template <int D, int RING, bool STREAM>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(RING <= 4 ? 2 : 1, RING <= 4 ? 8 : 1))) void k_attn_bf16(AttnArgs a) {
  constexpr int NC = D / 32;
  constexpr int NJ = D / 16;
  // the prefill launch (pages re-read: plain loads) runs on token groups (mq_col)
  constexpr bool MQ = !STREAM;
  // q rows of the chunk's later segments, [segment - 1][G][D]
  __shared__ __align__(16) uint16_t q_lds[kStageUnits * 64 * 8];
  // finished segments' softmax states, [segment][G][D] accumulators and
  // [segment][G] (m, l): (segments - 1) G D <= 8 kStageUnits * 64 by the plan
  __shared__ __align__(16) float st_acc[kStageUnits * 64 * 8];
  __shared__ float st_ml[kMaxSeg * kMaxGroup * 2];
  const int lane = threadIdx.x;
  const int col = lane & 15, quad = lane >> 4;
  const int G = a.group, Hkv = a.n_kv_heads;
  const int c = blockIdx.x / Hkv, g = blockIdx.x % Hkv;
  // Merge of the previous layer's split sequences (when a.mrg_acc is set):
  // items (sequence, kv-head, q-head) it = blockIdx.x, + gridDim.x, ... The
  // first item's loads are issued before anything else, so they arrive with
  // the first pages; the merge itself runs just before the page loop.
  const int n_mrg = a.mrg_acc ? a.n_seqs * Hkv * G : 0;
  MergeRegs<D> mr;
  int m_s = 0, m_g = 0, m_h = 0, m_n = 0;
  auto mrg_item = [&](int it) __attribute__((always_inline)) {
    m_s = it / (Hkv * G);
    m_g = (it / G) % Hkv;
    m_h = it % G;
    m_n = a.nparts[m_s];
    merge_load<D>(mr, a.mrg_acc, a.mrg_ml, (size_t)(m_s * Hkv + m_g) * a.split_stride, a.split_stride, G, m_h, 0,
                  lane);
  };
  if ((int)blockIdx.x < n_mrg) mrg_item(blockIdx.x);

  const int2 ci = a.chunk_info[c];
  const int nseg = ci.x, np = ci.y;  // 1 .. kMaxSeg segments, 1 .. kMaxSplitPages pages
  // the chunk's physical page ids and segment descriptors, lane k holding entry
  // k (read back with readlane; entries past the chunk's counts are never used)
  const int my_pid = a.work_pages[(size_t)c * kMaxSplitPages + lane];
  const int4* sd = a.seg + (size_t)c * kMaxSeg * 2;
  const int4 d0 = sd[2 * min(lane, kMaxSeg - 1)];
  const int4 d1 = sd[2 * min(lane, kMaxSeg - 1) + 1];
  const int4 e0 = sd[0], e1 = sd[1];  // segment 0, uniform loads
  int cur_s = e0.x, cur_poff = e0.z, cur_end = e0.w, cur_j = e1.x, cur_parts = e1.y;
  // Token groups: this lane's column ends mq_end_off keys before the group's
  // last token, so its keys in the segment end at min(segment end, keys of the
  // sequence - offset); a column may have none in a later split of its sequence.
  int col_end = cur_end;
  if constexpr (MQ) col_end = min(cur_end, e1.z - mq_end_off(a, cur_s, min(col, G - 1)));
  // (finite start in the grouped launch: a column without keys so far gives
  // weights 2^(-inf - m0) = 0 rather than NaN)
  constexpr float m0 = MQ ? -1e30f : kNegInf;

  const size_t q_layer = (size_t)a.layer * a.n_q_heads + (size_t)g * G;
  bf16x8 qop[NC];
  {
    // Columns past the group repeat its last head: their scores and outputs are
    // never stored, and the loads stay unconditional, so waiting for the page
    // ids below does not also wait for these.
    size_t qrow = (size_t)cur_s * a.n_layers * a.n_q_heads + q_layer + min(col, G - 1);
    if constexpr (MQ) {
      const MqCol m = mq_col(a, cur_s, g, min(col, G - 1));
      qrow = (size_t)m.row * a.n_q_heads + m.head;
    }
    const uint16_t* q = (const uint16_t*)a.q + qrow * D;
#pragma unroll
    for (int i = 0; i < NC; ++i) qop[i] = as_bf16x8(*(const uint4*)(q + 32 * i + 8 * quad));
  }
  const uint4* kp = (const uint4*)a.kpool;
  const uint4* vp = (const uint4*)a.vpool;
  const size_t lay = (size_t)a.layer * a.max_pages * Hkv + g;
  constexpr size_t tile16 = (size_t)kPage * D / 8;  // tile size in 16-byte units

  // Loads are issued unconditionally so that the wait before each page's use
  // leaves the next page in flight. Past the chunk's end they read physical page
  // 0 of the layer and kv-head, one tile that every wave's extra loads share, so
  // they stay cache hits although the page loads carry the streaming hint (the
  // chunk's own last page again missed the caches: +20 MB per launch); all of
  // their tokens are masked.
  auto load_page = [&](int i, uint4 (&kb)[NC], uint4 (&vb)[NC]) {
    const int phys = i < np ? __builtin_amdgcn_readlane(my_pid, min(i, 63)) : 0;
    const size_t t0 = (lay + (size_t)phys * Hkv) * tile16;
#pragma unroll
    for (int cc = 0; cc < NC; ++cc) {
      kb[cc] = ld_w<STREAM>(&kp[t0 + cc * 64 + lane]);
      vb[cc] = ld_w<STREAM>(&vp[t0 + cc * 64 + lane]);
    }
  };

  f32x4 acc[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  // Online softmax with a lazily moved reference: weights are 2^(z - m_ref) with
  // m_ref per head, shared by the head's four lanes. m_ref (and the accumulators)
  // only move when some score of the page exceeds m_ref + 8, so weights stay
  // <= 2^8 and the common page needs neither cross-lane traffic nor a rescale.
  float m_ref = m0, l_part = 0.f;
  int k = 0;
  int next_i0 = nseg > 1 ? sd[2].y : 0x7fffffff;

  // Write a finished segment, whose state is in LDS slot `slot`: the final
  // output when its sequence lies in this chunk alone, else its partial state
  // for the merge kernel, copied by all 64 lanes as whole contiguous lines
  // (the slot has the partial's [G][D] layout).
  auto emit = [&](int slot, int s, int part, int parts) __attribute__((always_inline)) {
    const float* sa = st_acc + slot * G * D;
    const float* sm = st_ml + slot * G * 2;
    if (parts == 1) {
      if (col >= G) return;
      const float inv = 1.0f / sm[2 * col + 1];
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const float4 v = *(const float4*)(sa + col * D + 16 * j + 4 * quad);
        write_o4<true, MQ>(a, s, g * G + col, 16 * j + 4 * quad, D,
                           make_float4(v.x * inv, v.y * inv, v.z * inv, v.w * inv));
      }
      return;
    }
    // partial state: the head's normalised output acc / l rounded to bf16 (a
    // convex combination of V rows, so bf16 keeps its range) plus (m, l) in fp32
    const size_t w = (size_t)(s * Hkv + g) * a.split_stride + part;
    uint16_t* dst = (uint16_t*)a.part_acc + w * G * D;
    for (int e = 8 * lane; e < G * D; e += 512) {
      const float l = sm[2 * (e / D) + 1];
      const float inv = l > 0.f ? 1.0f / l : 0.f;  // (a token-group column with no keys here: zeros)
      const float4 v0 = *(const float4*)(sa + e), v1 = *(const float4*)(sa + e + 4);
      uint4 pk;
      pk.x = f2bf(v0.x * inv) | (f2bf(v0.y * inv) << 16);
      pk.y = f2bf(v0.z * inv) | (f2bf(v0.w * inv) << 16);
      pk.z = f2bf(v1.x * inv) | (f2bf(v1.y * inv) << 16);
      pk.w = f2bf(v1.z * inv) | (f2bf(v1.w * inv) << 16);
      *(uint4*)(dst + e) = pk;
    }
    if (lane < 2 * G) a.part_ml[w * G * 2 + lane] = sm[lane];
  };
  auto reg_acc4 = [&](int j) __attribute__((always_inline)) {
    return make_float4(acc[j][0], acc[j][1], acc[j][2], acc[j][3]);
  };
  auto l_total = [&]() __attribute__((always_inline)) {
    float l_tot = l_part + __shfl_xor(l_part, 16);
    return l_tot + __shfl_xor(l_tot, 32);
  };
  // At a segment switch the finished state goes to LDS, not to memory: a store
  // inside the page loop would make every later wait of that iteration drain the
  // whole ring (stores and loads share the wave's memory counter). The states are
  // written out after the loop.
  auto save = [&](int slot) __attribute__((always_inline)) {
    const float l_tot = l_total();
    if (col < G) {
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        *(float4*)(st_acc + (slot * G + col) * D + 16 * j + 4 * quad) = reg_acc4(j);
      if (quad == 0) {
        st_ml[(slot * G + col) * 2] = m_ref;
        st_ml[(slot * G + col) * 2 + 1] = l_tot;
      }
    }
  };

  uint4 stg0, stg1, stg2, stg3;  // staged q units of later segments (filled after the ring starts)
  auto process = [&](int i, uint4 (&kc)[NC], uint4 (&vc)[NC]) __attribute__((always_inline)) {
    if (i == next_i0) {  // first page of the next segment
      save(k);
      if (k == 0) {  // units past the count land in unused LDS
        *(uint4*)(q_lds + 8 * lane) = stg0;
        *(uint4*)(q_lds + 8 * (lane + 64)) = stg1;
        *(uint4*)(q_lds + 8 * (lane + 128)) = stg2;
        *(uint4*)(q_lds + 8 * (lane + 192)) = stg3;
      }
      ++k;
      cur_s = __builtin_amdgcn_readlane(d0.x, k);
      cur_poff = __builtin_amdgcn_readlane(d0.z, k);
      cur_end = __builtin_amdgcn_readlane(d0.w, k);
      cur_j = __builtin_amdgcn_readlane(d1.x, k);
      cur_parts = __builtin_amdgcn_readlane(d1.y, k);
      next_i0 = k + 1 < nseg ? __builtin_amdgcn_readlane(d0.y, k + 1) : 0x7fffffff;
      col_end = cur_end;
      if constexpr (MQ)
        col_end = min(cur_end, __builtin_amdgcn_readlane(d1.z, k) - mq_end_off(a, cur_s, min(col, G - 1)));
      const uint16_t* qs = q_lds + ((k - 1) * G + min(col, G - 1)) * D + 8 * quad;
#pragma unroll
      for (int cc = 0; cc < NC; ++cc) qop[cc] = as_bf16x8(*(const uint4*)(qs + 32 * cc));
      m_ref = m0;
      l_part = 0.f;
#pragma unroll
      for (int j = 0; j < NJ; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    f32x4 sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int cc = 0; cc < NC; ++cc)
      sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kc[cc]), qop[cc], sc, 0, 0, 0);
    const int tb = (i + cur_poff) * kPage + 4 * quad;  // token of element r = 0 in the sequence
    float z[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) z[r] = (tb + r < col_end) ? sc[r] * a.scale_log2 : kNegInf;
    const float zmax = fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3]));
    if (__builtin_amdgcn_ballot_w64(zmax > m_ref + 8.0f) != 0) {
      float mx = fmaxf(zmax, __shfl_xor(zmax, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_ref, mx);
      const float alpha = exp2f(m_ref - m_new);
      l_part *= alpha;
#pragma unroll
      for (int j = 0; j < NJ; ++j) acc[j] *= alpha;
      m_ref = m_new;
    }
    uint32_t pb[4];
    float psum = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      pb[r] = f2bf(exp2f(z[r] - m_ref));
      psum += bf2f(pb[r]);   // normaliser uses exactly the weights fed to the MFMA
    }
    l_part += psum;
    s16x4 pop;
    pop[0] = (short)pb[0]; pop[1] = (short)pb[1]; pop[2] = (short)pb[2]; pop[3] = (short)pb[3];
    if ((i + cur_poff) * kPage + kPage > cur_end) {
      // Partial last page: slots past the segment's end hold stale or never-written
      // bits (or the next chunk's tokens). Their weights are 0, but 0 * NaN is NaN
      // inside the matrix core, so clear the V elements of those tokens (lane
      // elements r = 0..3 are the same tokens tb + r as its weights).
      const uint32_t m01 = (tb + 0 < cur_end ? 0x0000FFFFu : 0u) | (tb + 1 < cur_end ? 0xFFFF0000u : 0u);
      const uint32_t m23 = (tb + 2 < cur_end ? 0x0000FFFFu : 0u) | (tb + 3 < cur_end ? 0xFFFF0000u : 0u);
#pragma unroll
      for (int cc = 0; cc < NC; ++cc) {
        vc[cc].x &= m01; vc[cc].y &= m23; vc[cc].z &= m01; vc[cc].w &= m23;
      }
    }
#pragma unroll
    for (int cc = 0; cc < NC; ++cc) {
      const s16x4 va = __builtin_bit_cast(s16x4, make_uint2(vc[cc].x, vc[cc].y));
      const s16x4 vb = __builtin_bit_cast(s16x4, make_uint2(vc[cc].z, vc[cc].w));
      acc[2 * cc] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, pop, acc[2 * cc], 0, 0, 0);
      acc[2 * cc + 1] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vb, pop, acc[2 * cc + 1], 0, 0, 0);
    }
  };

  // RING-page register ring (4 at two waves per SIMD): the refill of page
  // i+RING-1 (into the buffer of page i-1, already consumed) is issued before
  // page i is consumed, so RING-1 pages are always in flight. The body is branch-free (a segment switch only touches
  // registers, LDS and stores) so that every iteration ends with the same loads
  // outstanding and the compiler's wait counts stay partial across the back
  // edge: pages past the chunk's end (the shared page 0, see load_page)
  // contribute nothing (all their tokens are masked).
  uint4 kr[RING][NC], vr[RING][NC];
  // the prologue keeps its issue order (the scheduler would otherwise reverse
  // it, and the wait at the loop head then has to drain every load)
#pragma unroll
  for (int j = 0; j < RING - 1; ++j) {
    load_page(j, kr[j], vr[j]);
    __builtin_amdgcn_sched_barrier(0);
  }
  // Later segments' q rows: 16-byte units u = ((k - 1) G + h) D/8 + d/8, spread
  // over lanes. Issued after the ring's first pages (loads complete in order, so
  // page 0 does not wait for them) and stored to LDS at the first switch.
  const int per_seg = G * (D / 8);
  const int n_units = (nseg - 1) * per_seg;
  // (unconditional loads: a unit past the count re-reads segment 0's first row)
  static_assert(kStageUnits == 4, "staging registers below");
  auto stage = [&](int r) __attribute__((always_inline)) {
    const int u = lane + 64 * r;
    const bool valid = u < n_units;
    const int kk = min(1 + u / per_seg, kMaxSeg - 1), rem = valid ? u % per_seg : 0;
    const int sk = valid ? __shfl(d0.x, kk) : e0.x;
    size_t qrow = (size_t)sk * a.n_layers * a.n_q_heads + q_layer + rem / (D / 8);
    if constexpr (MQ) {
      const MqCol m = mq_col(a, sk, g, rem / (D / 8));
      qrow = (size_t)m.row * a.n_q_heads + m.head;
    }
    return *(const uint4*)((const uint16_t*)a.q + qrow * D + 8 * (rem % (D / 8)));
  };
  stg0 = stage(0);
  stg1 = stage(1);
  stg2 = stage(2);
  stg3 = stage(3);
  for (int it = blockIdx.x; it < n_mrg; it += gridDim.x) {
    if (it != (int)blockIdx.x) mrg_item(it);
    merge_item<D>(a, mr, a.mrg_acc, a.mrg_ml, m_s, m_g, m_h, m_n, a.mrg_layer, false, lane);
  }
  for (int i = 0; i < np; i += RING) {
#pragma unroll
    for (int j = 0; j < RING; ++j) {
      load_page(i + j + RING - 1, kr[(j + RING - 1) % RING], vr[(j + RING - 1) % RING]);
      process(i + j, kr[j], vr[j]);
    }
  }
  // the saved segments, then the last one through slot 0 (LDS accesses of one
  // wave stay in order, so slot 0 is read out before it is overwritten)
  for (int kk = 0; kk < k; ++kk)
    emit(kk, __builtin_amdgcn_readlane(d0.x, kk), __builtin_amdgcn_readlane(d1.x, kk),
         __builtin_amdgcn_readlane(d1.y, kk));
  save(0);
  emit(0, cur_s, cur_j, cur_parts);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// fp32 caches (small/validation shapes): one wave per (chunk, kv-head) of the
// balanced plan, lanes over head dims (D <= 128), one token at a time, per-head
// online softmax in base 2; the chunk's segments one after another.
__global__ __launch_bounds__(64) void k_attn_f32(AttnArgs a, int D) {
  const int lane = threadIdx.x;
  const int G = a.group, Hkv = a.n_kv_heads;
  const int c = blockIdx.x / Hkv, g = blockIdx.x % Hkv;
  const int nseg = a.chunk_info[c].x;
  const bool has0 = lane < D, has1 = lane + 64 < D;
  const size_t tile = (size_t)kPage * D;
  const float* kp = (const float*)a.kpool;
  const float* vp = (const float*)a.vpool;
  const size_t lay = (size_t)a.layer * a.max_pages * Hkv + g;
  for (int k = 0; k < nseg; ++k) {
    const int4 d0 = a.seg[((size_t)c * kMaxSeg + k) * 2], d1 = a.seg[((size_t)c * kMaxSeg + k) * 2 + 1];
    const int s = d0.x, tok_end = d0.w;
    const float* q = (const float*)a.q + (((size_t)s * a.n_layers + a.layer) * a.n_q_heads + (size_t)g * G) * D;
    float qv[kMaxGroup][2], m[kMaxGroup], l[kMaxGroup], acc[kMaxGroup][2];
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h) {
      qv[h][0] = (h < G && has0) ? q[h * D + lane] : 0.f;
      qv[h][1] = (h < G && has1) ? q[h * D + lane + 64] : 0.f;
      m[h] = kNegInf; l[h] = 0.f; acc[h][0] = 0.f; acc[h][1] = 0.f;
    }
    const int32_t* pt = a.page_table + (size_t)s * a.maxpps;
    for (int tok = (d0.y + d0.z) * kPage; tok < tok_end; ++tok) {
      const size_t base = (lay + (size_t)pt[tok / kPage] * Hkv) * tile + (size_t)(tok % kPage) * D;
      const float k0 = has0 ? kp[base + lane] : 0.f, k1 = has1 ? kp[base + lane + 64] : 0.f;
      const float v0 = has0 ? vp[base + lane] : 0.f, v1 = has1 ? vp[base + lane + 64] : 0.f;
#pragma unroll
      for (int h = 0; h < kMaxGroup; ++h) {
        if (h >= G) continue;  // (G is uniform: the rest are skipped too)
        const float z = wave_sum(qv[h][0] * k0 + qv[h][1] * k1) * a.scale_log2;
        const float mn = fmaxf(m[h], z);
        const float al = exp2f(m[h] - mn), pz = exp2f(z - mn);
        l[h] = l[h] * al + pz;
        acc[h][0] = acc[h][0] * al + pz * v0;
        acc[h][1] = acc[h][1] * al + pz * v1;
        m[h] = mn;
      }
    }
    if (d1.y == 1) {  // the sequence lies in this chunk alone: final output
#pragma unroll
      for (int h = 0; h < kMaxGroup; ++h) {
        if (h >= G) continue;  // (G is uniform: the rest are skipped too)
        const float inv = 1.0f / l[h];
        const int head = g * G + h;
        const size_t xo = (size_t)s * a.n_q_heads * D + (size_t)head * D;
        const size_t ao = (((size_t)s * a.n_layers + a.layer) * a.n_q_heads + head) * D;
        for (int cc = 0; cc < 2; ++cc) {
          const int d = lane + 64 * cc;
          if (d >= D) break;
          const float o = acc[h][cc] * inv;
          ((float*)a.x_out)[xo + d] = o;
          if (a.attn_out) a.attn_out[ao + d] = o;
          if (a.is_last_layer && a.hidden_out) a.hidden_out[xo + d] = o;
        }
      }
      continue;
    }
    const size_t w = (size_t)(s * Hkv + g) * a.split_stride + d1.x;
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h) {
      if (h >= G) continue;
      if (has0) a.part_acc[(w * G + h) * D + lane] = acc[h][0];
      if (has1) a.part_acc[(w * G + h) * D + lane + 64] = acc[h][1];
      if (lane == 0) {
        a.part_ml[(w * G + h) * 2] = m[h];
        a.part_ml[(w * G + h) * 2 + 1] = l[h];
      }
    }
  }
}

// --------------------------------------------------- LM head: sum of squares

__device__ __forceinline__ float sumsq8(bf16x8 v) {
  const uint4 u = __builtin_bit_cast(uint4, v);
  float s = 0.f;
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float lo = __uint_as_float(w[i] << 16), hi = __uint_as_float(w[i] & 0xFFFF0000u);
    s += lo * lo + hi * hi;
  }
  return s;
}

// ------------------------------------------------------ argmax helpers (Eq. 3)

struct Top2 {
  float v1; int i1; int k1; float v2; int i2;
};

// order: higher score first, lower token id on equal scores
__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

__device__ __forceinline__ Top2 merge(const Top2& A, const Top2& B) {
  // winner's best, then the better of the winner's second and the loser's best
  // (written with selects only, so the candidates stay in registers)
  const bool af = better(A.v1, A.i1, B.v1, B.i1);
  const float wv2 = af ? A.v2 : B.v2, lv1 = af ? B.v1 : A.v1;
  const int wi2 = af ? A.i2 : B.i2, li1 = af ? B.i1 : A.i1;
  const bool w2 = better(wv2, wi2, lv1, li1);
  Top2 R;
  R.v1 = af ? A.v1 : B.v1;
  R.i1 = af ? A.i1 : B.i1;
  R.k1 = af ? A.k1 : B.k1;
  R.v2 = w2 ? wv2 : lv1;
  R.i2 = w2 ? wi2 : li1;
  return R;
}

__device__ __forceinline__ Top2 shfl_top2(const Top2& x, int o) {
  Top2 y;
  y.v1 = __shfl_xor(x.v1, o); y.i1 = __shfl_xor(x.i1, o); y.k1 = __shfl_xor(x.k1, o);
  y.v2 = __shfl_xor(x.v2, o); y.i2 = __shfl_xor(x.i2, o);
  return y;
}

// Two-level argmax over a block of NW waves: a wave merges its lanes' candidates
// with shuffles, the block merges its waves through LDS. Deterministic for any
// merge order: "better" is a total order on (score, token).
template <int NW>
__device__ Top2 block_top2(Top2 c) {
  __shared__ Top2 red[NW];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) c = merge(c, shfl_top2(c, o));
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[wave] = c;
  __syncthreads();
  Top2 r = red[0];
#pragma unroll
  for (int i = 1; i < NW; ++i) r = merge(r, red[i]);
  __syncthreads();
  return r;
}

// Eq. 2 and the best two tokens per query over a block's logits tile (the LM
// head's fused epilogue). The NC columns are vocabulary ids v0 .. v0+NC-1; row m
// of column j is read through at(m, j). The block's NW waves form groups of NC
// threads, one column per thread, and the groups take the queries in turn; the
// experts' scores are read eight at a time so their LDS latencies overlap
// (rows past the query's last are read too, clamped to the tile's last row
// max_row, and not used: unconditional reads issue back to back). The
// arithmetic is k_fuse's, in the same order and without contraction, so the
// result is bit-identical to materialising the logits and fusing them
// afterwards. Writes fuse_part[b][blk] for every query b.
template <int NW, int NC, typename At>
__device__ void fuse_tile(const LmArgs& a, int v0, int blk, At at, int max_row) {
#pragma clang fp contract(off)
  constexpr int NG = 64 * NW / NC;  // thread groups (queries in flight)
  constexpr int WG = NC / 64;       // waves per group
  static_assert(NG >= 1 && NC % 64 == 0, "whole waves per group");
  __shared__ Top2 red[NG][WG];
  // beta and prior of every expert, staged once (fused launches have < 288 experts)
  __shared__ float cb[32 * kLmRowsMTW], pr[32 * kLmRowsMTW];
  const int n_exp = a.query_exp0[a.n_queries];
  for (int i = threadIdx.x; i < n_exp; i += 64 * NW) {
    cb[i] = a.beta[i];
    pr[i] = a.prior[i];
  }
  __syncthreads();
  const int g = threadIdx.x / NC, j = threadIdx.x % NC, wg = j >> 6;
  const int v = v0 + j;
  for (int b0 = 0; b0 < a.n_queries; b0 += NG) {
    // one query per wave: uniform, so its row range, beta and prior come by scalar loads
    const int b = __builtin_amdgcn_readfirstlane(b0 + g);
    Top2 c{kNegInf, 0x7FFFFFFF, 0, kNegInf, 0x7FFFFFFF};
    if (b < a.n_queries && v < a.V) {
      const int s0 = a.query_seq0[b];
      const int N = a.query_seq0[b + 1] - s0 - 1;
      const int e0 = a.query_exp0[b];
      const float sa = at(s0, j);
      float best = kNegInf;
      int bk = 0;
      for (int kb = 1; kb <= N; kb += 8) {
        float x[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) x[u] = at(min(s0 + kb + u, max_row), j);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          // past the query's last expert: an in-bounds entry, the result unused
          const int k = kb + u, ei = min(e0 + k - 1, 32 * kLmRowsMTW - 1);
          const float beta = cb[ei];
          const float coef = 1.0f + beta;
          const float t1 = coef * x[u];
          const float t2 = beta * sa;
          const float val = (t1 - t2) + pr[ei];
          if (k <= N && val > best) { best = val; bk = k; }
        }
      }
      c.v1 = best; c.i1 = v; c.k1 = bk;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) c = merge(c, shfl_top2(c, o));
    if ((threadIdx.x & 63) == 0) red[g][wg] = c;
    __syncthreads();
    if (j == 0 && b < a.n_queries) {
      Top2 r = red[g][0];
#pragma unroll
      for (int i = 1; i < WG; ++i) r = merge(r, red[g][i]);
      float* p = a.fuse_part + ((size_t)b * a.fuse_nblk + blk) * 5;
      p[0] = r.v1; p[1] = __int_as_float(r.i1); p[2] = __int_as_float(r.k1);
      p[3] = r.v2; p[4] = __int_as_float(r.i2);
    }
    __syncthreads();
  }
}

// Rows a block reads past a query's last one in the many-row LM head's fused
// epilogue (whole 16-byte groups of 4 rows, two groups per step).
constexpr int kWideOverRead = 40;

// What the many-row LM head's fused epilogue reads besides its tile, staged in
// LDS at the start of the launch (an empty struct without the epilogue): row
// scales, beta and prior per row (each expert's at its row; amateur rows and
// rows past M hold stale values that are never used) and the queries' first
// rows.
template <bool FUSED>
struct WideEpi {
  __align__(16) float beta_row[kLmWideMaxRows + kWideOverRead];
  __align__(16) float prior_row[kLmWideMaxRows + kWideOverRead];
  float rho[kLmWideMaxRows];
  int qs[kLmWideMaxRows / 2 + 1];
};
template <>
struct WideEpi<false> {};

// Eq. 2 for the experts k0 .. k0 + 3 (scores x, beta b, prior p of their rows;
// sa the amateur's score), keeping the best over those with 1 <= k <= N, the
// lower k on equal scores. k_fuse's arithmetic in its order, no contraction.
__device__ __forceinline__ void eq2_rows4(const float4 x, const float4 b, const float4 p, float sa, int k0, int N,
                                          float& best, int& bk) {
#pragma clang fp contract(off)
  const float xv[4] = {x.x, x.y, x.z, x.w}, bv[4] = {b.x, b.y, b.z, b.w}, pv[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int k = k0 + q;
    const float coef = 1.0f + bv[q];
    const float t1 = coef * xv[q];
    const float t2 = bv[q] * sa;
    const float val = (t1 - t2) + pv[q];
    if (k >= 1 && k <= N && val > best) {
      best = val;
      bk = k;
    }
  }
}

// ------------------------------------------------------------------- LM head

// Packed LM-head layout (bf16). W [V][K] is re-laid once into 2 KiB tiles, one
// per (16-row vocab block vb, 64-wide k step ks); tile (vb, ks) sits at tile
// index vb * t_vb + ks * t_ks ([vb][ks]: t_vb = K/64, t_ks = 1; the LM head's
// k-major order: t_vb = 1, t_ks = vocab blocks). Inside
// a tile, half h (0, 1) and lane l = col + 16*quad hold the 8 elements
// W[16*vb + col][64*ks + 16*quad + 8*h .. +7]: each half is exactly the A operand
// of one v_mfma_f32_16x16x32_bf16, read as one contiguous 1 KiB wave load.
// Rows past V are zero.
// Row tile vb of the source goes to vocab block vb * stride + offset of wp (the
// decoder projections interleave or concatenate several matrices this way).
__global__ __launch_bounds__(256) void k_pack_w_bf16(const uint16_t* __restrict__ w, uint16_t* __restrict__ wp,
                                                     int V, int K, int stride, int offset, size_t t_vb,
                                                     size_t t_ks) {
  const int KS = K / 64;
  const size_t n16 = (size_t)((V + 15) / 16) * KS * 2 * 64;  // 16-byte units of the packed matrix
  for (size_t u = blockIdx.x * (size_t)blockDim.x + threadIdx.x; u < n16; u += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(u & 63);
    const size_t t = u >> 6;
    const int h = (int)(t & 1);
    const size_t tile = t >> 1;
    const int ks = (int)(tile % KS);
    const int vb = (int)(tile / KS);
    const int v = 16 * vb + (lane & 15);
    const int k = 64 * ks + 16 * (lane >> 4) + 8 * h;
    uint4 val = make_uint4(0u, 0u, 0u, 0u);
    if (v < V) val = *(const uint4*)(w + (size_t)v * K + k);
    const size_t dst = ((((size_t)vb * stride + offset) * t_vb + ks * t_ks) * 2 + h) * 64 + lane;
    *(uint4*)(wp + dst * 8) = val;
  }
}

// logits[m][v] = rho_m * sum_k x[m][k] W[v][k] on the matrix cores:
// C^T[16 vocab x 16 rows] += W[16 x 32] X^T[32 x 16] (v_mfma_f32_16x16x32_bf16).
// A wave owns VT consecutive 16-row vocab blocks and streams their packed tiles
// (contiguous 1 KiB loads) exactly once per 16*NT rows of x, through a 3-stage
// register ring (two 64-wide k steps in flight); the x operands (a few hundred
// KiB, L2-resident) are loaded one step ahead.
// rho (the RMS scale) is accumulated from the same x operands.
template <int VT, int NT, bool FUSED, bool STREAM>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_lmhead_bf16(LmArgs a) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, quad = lane >> 4;
  // Work-groups are dealt to the 8 XCDs round-robin. With R = a.row_groups > 1,
  // the R row groups of one vocab chunk are consecutive work-groups of the same
  // XCD, so they stream the same W tiles together and all but the first read
  // them from that XCD's L2.
  const int R = max(a.row_groups, 1);
  int chunk = blockIdx.x, rg = 0;
  if (R > 1) {
    const int xcd = blockIdx.x % 8, i = blockIdx.x / 8;
    chunk = xcd + 8 * (i / R);
    rg = i % R;
  }
  const int vb0 = (chunk * 4 + wave) * VT;   // first 16-row vocab block of the wave
  const int nvb = (a.V + 15) / 16;
  if (!FUSED && vb0 >= nvb) return;  // (fused: every wave reaches the block's barriers)
  const int K = a.K, KS = K / 64;
  const uint16_t* X = (const uint16_t*)a.x;
  // W tile addresses: a wave-uniform 64-bit base (scalar registers) plus the
  // lane's 16 bytes, so the ring's loads cost no per-lane pointer registers
  const char* Wb = (const char*)a.w;
  const uint32_t lane16 = 16u * lane;
  size_t wvb[VT];
#pragma unroll
  for (int vt = 0; vt < VT; ++vt)
    wvb[vt] = (size_t)__builtin_amdgcn_readfirstlane(min(vb0 + vt, nvb - 1)) * a.w_vb * 16;
  for (int m0 = rg * 16 * NT; m0 < a.M; m0 += 16 * NT * R) {
    f32x4 acc[VT][NT];
    float ss[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      ss[nt] = 0.f;
#pragma unroll
      for (int vt = 0; vt < VT; ++vt) acc[vt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const uint16_t* xrow[NT];
#pragma unroll
    // rows past M (padding of the last tile, never stored) read row M - 1: the
    // same lines as that row, not 15 more per step
    for (int nt = 0; nt < NT; ++nt) xrow[nt] = X + (size_t)min(m0 + 16 * nt + col, a.M - 1) * K + 16 * quad;
    struct WS { uint4 w[VT][2]; };
    struct XS { uint4 x[NT][2]; };
    auto load_w = [&](WS& S, int ks) {
      ks = min(ks, KS - 1);  // past the end: the last step again (cache hit), keeps the ring branch-free
      const size_t kso = (size_t)ks * a.w_ks * 16;
#pragma unroll
      for (int vt = 0; vt < VT; ++vt) {
        const char* base = Wb + wvb[vt] + kso;
        S.w[vt][0] = ld_w<STREAM>((const uint4*)(base + lane16));
        S.w[vt][1] = ld_w<STREAM>((const uint4*)(base + 1024 + lane16));
      }
    };
    auto load_x = [&](XS& S, int ks) {
      ks = min(ks, KS - 1);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        S.x[nt][0] = *(const uint4*)(xrow[nt] + ks * 64);
        S.x[nt][1] = *(const uint4*)(xrow[nt] + ks * 64 + 8);
      }
    };
    auto step = [&](const WS& A, const XS& B) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        ss[nt] += sumsq8(as_bf16x8(B.x[nt][0])) + sumsq8(as_bf16x8(B.x[nt][1]));
#pragma unroll
        for (int vt = 0; vt < VT; ++vt) {
          acc[vt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(A.w[vt][0]), as_bf16x8(B.x[nt][0]),
                                                                acc[vt][nt], 0, 0, 0);
          acc[vt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(A.w[vt][1]), as_bf16x8(B.x[nt][1]),
                                                                acc[vt][nt], 0, 0, 0);
        }
      }
    };
    // W: three-stage ring (two 64-wide k steps in flight while one is consumed);
    // x: two stages (one step ahead). Each step's x is issued before the W of
    // two steps later: vector loads retire in order, so waiting for x never
    // waits for W that is not needed yet. The pattern repeats every 6 steps.
    WS w0, w1, w2;
    XS xa, xb;
    load_x(xa, 0);
    load_w(w0, 0);
    load_w(w1, 1);
    for (int ks = 0; ks < KS; ks += 6) {
      load_x(xb, ks + 1); load_w(w2, ks + 2); step(w0, xa);
      load_x(xa, ks + 2); load_w(w0, ks + 3); if (ks + 1 < KS) step(w1, xb);
      load_x(xb, ks + 3); load_w(w1, ks + 4); if (ks + 2 < KS) step(w2, xa);
      load_x(xa, ks + 4); load_w(w2, ks + 5); if (ks + 3 < KS) step(w0, xb);
      load_x(xb, ks + 5); load_w(w0, ks + 6); if (ks + 4 < KS) step(w1, xa);
      load_x(xa, ks + 6); load_w(w1, ks + 7); if (ks + 5 < KS) step(w2, xb);
    }
    if constexpr (FUSED) {
      // logits tile of the block (rows x 256 columns, rows padded by 16 bytes
      // against bank conflicts), then Eq. 2 per column (one row group: m0 = 0)
      constexpr int LD = 64 * VT + 4;
      __shared__ __align__(16) float tile[16 * NT * LD];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        float t = ss[nt] + __shfl_xor(ss[nt], 16);
        t += __shfl_xor(t, 32);
        const int m = 16 * nt + col;
        if (m >= a.M) continue;
        const float rho = a.rho_in ? a.rho_in[m] : a.rms ? 1.0f / sqrtf(t / (float)K + 1e-5f) : 1.0f;
#pragma unroll
        for (int vt = 0; vt < VT; ++vt) {
          const f32x4 cc = acc[vt][nt];
          *(float4*)(tile + m * LD + 64 * wave + 16 * vt + 4 * quad) =
              make_float4(cc[0] * rho, cc[1] * rho, cc[2] * rho, cc[3] * rho);
        }
      }
      __syncthreads();
      fuse_tile<4, 64 * VT>(a, chunk * 256, chunk, [&](int m, int j) { return tile[m * LD + j]; }, 16 * NT - 1);
      return;  // fused: at most 16 NT rows, a single row group
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      float t = ss[nt] + __shfl_xor(ss[nt], 16);
      t += __shfl_xor(t, 32);
      const int m = m0 + 16 * nt + col;
      if (m >= a.M) continue;
      const float rho = a.rho_in ? a.rho_in[m] : a.rms ? 1.0f / sqrtf(t / (float)K + 1e-5f) : 1.0f;
#pragma unroll
      for (int vt = 0; vt < VT; ++vt) {
        const int v = 16 * (vb0 + vt) + 4 * quad;
        float* out = a.logits + (size_t)m * a.V + v;
        const f32x4 cc = acc[vt][nt];
        if (v + 3 < a.V && (a.V & 3) == 0) {
          *(float4*)out = make_float4(cc[0] * rho, cc[1] * rho, cc[2] * rho, cc[3] * rho);
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (v + r < a.V) out[r] = cc[r] * rho;
        }
      }
    }
  }
}

// LM head for many rows: W is streamed exactly once for all M <= 32 MTW rows.
// A block of WPB waves owns WPB/2 * VTW consecutive 16-row vocab blocks; wave w takes
// vocab blocks [VTW (w/2), +VTW) and the row tiles w%2, w%2 + 2, ... (interleaved,
// so the two halves stay balanced for any M). The hidden dimension is walked in
// stages of 64 KB columns. For every stage the block stages the x slice of all
// rows in LDS (double buffered, in the lanes' B-operand order so each wave reads
// it conflict-free), filled by all 512 threads with coalesced row pieces; each
// wave streams its own packed W tiles straight from HBM through a 2-slot
// register ring refilled right after each stage's products; the next x slice is
// issued before that refill, so waiting for x never waits for W that is not
// due, and long stages keep each W load a full stage ahead of its use. The
// staging threads also accumulate every row's sum of squares (RMS scale).
template <int VTW, int MTW, int KB, int WPB, bool FUSED>
__global__ __launch_bounds__(64 * WPB) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_lmhead_rows_bf16(LmArgs a) {
  constexpr int NTH = 64 * WPB;          // threads per block
  constexpr int MT = 2 * MTW;            // row tiles the kernel holds
  constexpr int SUB = MT * 128;          // 16-byte x units of one 64-wide k step
  constexpr int UNITS = SUB * KB;        // ... of one stage
  constexpr int UPT = (UNITS + NTH - 1) / NTH;
  constexpr int PIECES = 8 * KB;         // 16-byte pieces of a row's stage slice
  // Row-major stage slice, rows padded by one 16-byte unit (odd stride): the
  // coalesced staging stores (consecutive pieces of a row) and the B-operand
  // reads (16 rows x 4 pieces per wave load) both spread over all banks. (The
  // slice in B-operand order made each wave's stores hit the same banks 8 to
  // 16 times over: bank conflicts took 70% of the LDS cycles.)
  constexpr int RS = PIECES + 1;
  __shared__ __align__(16) uint4 xs[2][MT * 16 * RS];
  __shared__ float rho_s[MT * 16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane & 15, quad = lane >> 4;
  const int K = a.K, KS = K / (64 * KB), M = a.M;
  const int nt = (M + 15) / 16;          // row tiles in use
  const int n_units = nt * 16 * PIECES;  // units of the rows in use, per stage
  const int nvb = (a.V + 15) / 16;
  const int rh = wave & 1;
  const int vb0 = (blockIdx.x * (WPB / 2) + (wave >> 1)) * VTW;
  const uint4* Wp = (const uint4*)a.w;
  const uint16_t* X = (const uint16_t*)a.x;
  const uint4* wt[VTW];
#pragma unroll
  for (int vt = 0; vt < VTW; ++vt) wt[vt] = Wp + (size_t)min(vb0 + vt, nvb - 1) * a.w_vb + lane;

  // staging: thread unit v = tid + NTH j is row v / PIECES, 16-byte piece v % PIECES
  // of its stage slice (PIECES consecutive threads read one contiguous row piece);
  // unit j of a thread is NTH / PIECES rows below unit 0
  static_assert(NTH % (16 * PIECES) == 0, "whole tiles per staging round");
  constexpr int ROWS_J = NTH / PIECES;
  const int row0 = tid / PIECES, pc = tid % PIECES;
  // (x holds whole 16-row tiles: the callers' row buffers are padded to them)
  const uint16_t* xsrc = X + (size_t)row0 * K + 8 * pc;
  const int xdst = row0 * RS + pc;
  float ss[UPT];
#pragma unroll
  for (int j = 0; j < UPT; ++j) ss[j] = 0.f;
  uint4 xr[UPT];
  auto load_x = [&](int ks) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < UPT; ++j)
      if (tid + NTH * j < n_units) xr[j] = *(const uint4*)(xsrc + (size_t)j * ROWS_J * K + ks * 64 * KB);
  };
  auto store_x = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < UPT; ++j)
      if (tid + NTH * j < n_units) {
        xs[buf][xdst + j * ROWS_J * RS] = xr[j];
        ss[j] += sumsq8(as_bf16x8(xr[j]));
      }
  };
  struct WS { uint4 w[VTW][KB][2]; };
  auto load_w = [&](WS& S, int ks) __attribute__((always_inline)) {
    ks = min(ks, KS - 1);  // past the end: the last stage again (cache hit)
#pragma unroll
    for (int vt = 0; vt < VTW; ++vt)
#pragma unroll
      for (int sb = 0; sb < KB; ++sb) {
        S.w[vt][sb][0] = ld_w<true>(&wt[vt][(size_t)(ks * KB + sb) * a.w_ks]);
        S.w[vt][sb][1] = ld_w<true>(&wt[vt][(size_t)(ks * KB + sb) * a.w_ks + 64]);
      }
  };
  f32x4 acc[VTW][MTW];
#pragma unroll
  for (int i = 0; i < MTW; ++i)
#pragma unroll
    for (int vt = 0; vt < VTW; ++vt) acc[vt][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto step = [&](const WS& A, int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int sb = 0; sb < KB; ++sb)
#pragma unroll
      for (int i = 0; i < MTW; ++i) {
        const int t = 2 * i + rh;
        if (t < nt) {
          // lane (col, quad): row 16 t + col, elements 64 sb + 16 quad + 8 h .. + 7
          const uint4* xp = &xs[buf][(16 * t + col) * RS + 8 * sb + 2 * quad];
          const bf16x8 b0 = as_bf16x8(xp[0]);
          const bf16x8 b1 = as_bf16x8(xp[1]);
#pragma unroll
          for (int vt = 0; vt < VTW; ++vt) {
            acc[vt][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(A.w[vt][sb][0]), b0, acc[vt][i], 0, 0, 0);
            acc[vt][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(A.w[vt][sb][1]), b1, acc[vt][i], 0, 0, 0);
          }
        }
      }
  };
  // One stage with a two-slot W ring: issue x of ks+1, multiply stage ks, refill
  // the consumed slot with W of ks+2, publish x of ks+1. The refill is younger
  // than x of ks+1, so publishing x waits for W of ks+1 (used next) but not ks+2.
  auto sub = [&](int ks, WS& use) __attribute__((always_inline)) {
    if (ks >= KS) return;  // uniform
    if (ks + 1 < KS) load_x(ks + 1);
    step(use, ks & 1);
    load_w(use, ks + 2);
    if (ks + 1 < KS) store_x((ks + 1) & 1);
    __syncthreads();
  };
  WS w0, w1;
  load_x(0);
  store_x(0);
  load_w(w0, 0);
  load_w(w1, 1);
  __syncthreads();
  for (int ks = 0; ks < KS; ks += 2) {
    sub(ks, w0);
    sub(ks + 1, w1);
  }
  // RMS scale per row: the PIECES threads of a row are consecutive lanes
#pragma unroll
  for (int j = 0; j < UPT; ++j) {
    float t = ss[j];
#pragma unroll
    for (int o = 1; o < PIECES; o <<= 1) t += __shfl_xor(t, o);
    const int v = tid + NTH * j;
    if (v < n_units && v % PIECES == 0)
      rho_s[v / PIECES] = a.rho_in ? a.rho_in[v / PIECES] : a.rms ? 1.0f / sqrtf(t / (float)K + 1e-5f) : 1.0f;
  }
  __syncthreads();
  if constexpr (FUSED) {
    // logits tile of the block in the (now free) x buffers: rows x 128 columns,
    // float4 groups XOR-swizzled by row against bank conflicts; then Eq. 2 per column
    constexpr int NC = WPB / 2 * VTW * 16;  // columns of the block
    static_assert(NC == 128 && 2 * (MT * 16 * RS) * 4 >= 32 * MTW * NC, "tile fits the x buffers");
    float* tile = (float*)&xs[0][0];
    auto at = [&](int m, int j) { return tile[m * NC + ((((j >> 2) ^ (m & 31)) << 2) | (j & 3))]; };
#pragma unroll
    for (int i = 0; i < MTW; ++i) {
      const int m = 16 * (2 * i + rh) + col;
      if (m >= M) continue;
      const float rho = rho_s[m];
#pragma unroll
      for (int vt = 0; vt < VTW; ++vt) {
        const f32x4 cc = acc[vt][i];
        const int c4 = 8 * (wave >> 1) + 4 * vt + quad;
        *(float4*)(tile + m * NC + ((c4 ^ (m & 31)) << 2)) =
            make_float4(cc[0] * rho, cc[1] * rho, cc[2] * rho, cc[3] * rho);
      }
    }
    __syncthreads();
    fuse_tile<WPB, NC>(a, blockIdx.x * NC, blockIdx.x, at, 32 * MTW - 1);
    return;
  }
#pragma unroll
  for (int i = 0; i < MTW; ++i) {
    const int m = 16 * (2 * i + rh) + col;
    if (m >= M) continue;
    const float rho = rho_s[m];
#pragma unroll
    for (int vt = 0; vt < VTW; ++vt) {
      if (vb0 + vt >= nvb) continue;
      const int v = 16 * (vb0 + vt) + 4 * quad;
      float* out = a.logits + (size_t)m * a.V + v;
      const f32x4 cc = acc[vt][i];
      if (v + 3 < a.V && (a.V & 3) == 0) {
        *(float4*)out = make_float4(cc[0] * rho, cc[1] * rho, cc[2] * rho, cc[3] * rho);
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (v + r < a.V) out[r] = cc[r] * rho;
      }
    }
  }
}

// s_waitcnt that waits for the vector-memory counter only (vmcnt <= N); the
// expcnt / lgkmcnt fields are left at their "no wait" maxima.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt has 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

typedef __attribute__((address_space(3))) void lds_void;


// The many-row LM head's B operands, laid out in advance: x [M][K] bf16
// (row-major) into xp [K/64][MTP][2][64] 16-byte units, unit (ks, t, h, lane)
// holding x[16t + lane%16][64ks + 16(lane/16) + 8h .. +7], so that each
// (64-wide k step, 16-row tile, half) operand is one contiguous 1 KiB; rows
// M .. 16 MTP - 1 are zero. Also rho[m] = 1/sqrt(mean(x[m]^2) + 1e-5) (or 1
// without RMS) from the same reads. One wave per row, 16-byte loads.
__global__ __launch_bounds__(256) void k_pack_x(const uint16_t* __restrict__ x, int M, int K, int MTP, int rms,
                                                uint4* __restrict__ xp, float* __restrict__ rho) {
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (m >= 16 * MTP) return;
  const int t = m >> 4, col = m & 15;
  float ss = 0.f;
  for (int k = 8 * lane; k < K; k += 512) {
    const uint4 v = m < M ? *(const uint4*)(x + (size_t)m * K + k) : make_uint4(0u, 0u, 0u, 0u);
    ss += sumsq8(as_bf16x8(v));
    const int ks = k >> 6, kk = k & 63, quad = kk >> 4, h = (kk >> 3) & 1;
    xp[(((size_t)ks * MTP + t) * 2 + h) * 64 + col + 16 * quad] = v;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o);
  if (lane == 0 && m < M) rho[m] = rms ? 1.0f / sqrtf(ss / (float)K + 1e-5f) : 1.0f;
}

// Compile-time loop: f(integral_constant<int, i>) for i = 0 .. N-1, in order.
template <typename F, size_t... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::index_sequence<I...>) {
  (f(std::integral_constant<int, (int)I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_index_sequence<N>{});
}

// The many-row LM head's wait at the end of step s: vector loads retire in
// order, and half step h (relative to 2s) issues W(2s + h + lead) and then, at
// even h, x(s + h/2 + xl) (xb loads). Step s + 1 needs x(s + 1) and
// W(2s + 2), W(2s + 3); the result is the number of loads issued after the
// later of those two (w loads per half step), which may stay in flight.
constexpr int lmhead_wide_wait(int lead, int xl, int xb, int w) {
  const int hw = 3 - lead, hx = 2 - 2 * xl;  // half steps that issue W(2s + 3) and x(s + 1)
  int n = 0, from = 0;
  if (hw > hx) {
    n = (hw % 2 == 0) ? xb : 0;  // the x issued after W in half step hw
    from = hw + 1;
  } else {
    from = hx + 1;
  }
  for (int h = from; h <= 1; ++h) n += w + ((h % 2 == 0) ? xb : 0);
  return n;
}
static_assert(lmhead_wide_wait(7, 3, 5, 2) == 20 && lmhead_wide_wait(3, 3, 5, 4) == 9 &&
                  lmhead_wide_wait(15, 7, 2, 2) == 38,
              "wait counts");

// LM head for 49..288 rows with W read once: logits[m][v] = rho_m sum_k x[m][k] W[v][k]
// (x packed by k_pack_x, rho precomputed) on the matrix cores,
// C^T[16 vocab x 16 rows] += W[16 x 32] X^T[32 x 16] (v_mfma_f32_16x16x32_bf16).
// A block of 8 waves (two per SIMD) owns 256 vocabulary rows; wave w computes
// vocab rows 32w .. 32w + 31 of them (two 16-row tiles) for all MTP 16-row
// tiles of x (acc: 2 x MTP x 4 registers), so every W byte is loaded by exactly
// one wave. The products are cheap next to the weight stream, which they must
// hide, so both operands are fetched far ahead. The hidden dimension is walked
// in 32-wide half steps h, with NS = 4 LDS stages of x (8 when x has at most
// 128 rows, its stages then being small) and a W ring of WR = 2 NS slots:
//   - W of half step h + WR - 1 goes into slot (h + WR - 1) % WR of a register
//     ring (two tiles, 8 registers a slot);
//   - at even h the packed x of 64-wide step h/2 + NS - 1 goes from memory
//     straight into LDS stage (h/2 + NS - 1) % NS (buffer loads with the LDS
//     flag, no registers), the eight waves loading an eighth of its 1 KiB
//     operands each; x is fetched as far ahead as W because vector loads
//     retire in order, so waiting for an x issued after a W waits for that W;
//   - the 2 x MTP products of h read their B operands from LDS stage
//     (h/2) % NS, three tiles ahead of their use, each feeding two products;
//   - at odd h the wave waits until its loads of the next step's x and W have
//     landed, leaving every later load in flight, and meets the other waves
//     at a barrier, after which the next stage holds every wave's loads.
// Scheduling barriers keep each half step's loads ahead of its products. Loads
// past the end re-read the last step (in bounds, never used). FUSED: Eq. 2 and
// the slice argmax in the epilogue, in four passes of 64 columns through the
// (then free) LDS stages, with the row scales, beta and prior by row and the
// queries' first rows staged in LDS at the start.
template <int MTH, int NS, bool FUSED>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_lmhead_wide_bf16(LmArgs a) {
  static_assert(NS == 4 || NS == 8, "x stages");
  constexpr int MTP = 2 * MTH;           // 16-row tiles of the packed x
  constexpr int XU = 2 * MTP;            // 1 KiB B operands of one x stage (tiles x 2 halves)
  constexpr int XB = (XU + 7) / 8;       // of which each wave loads (the last one twice over if XU % 8 != 0)
  constexpr int WR = 2 * NS, LEAD = WR - 1;  // W ring slots; half steps of W in flight
  constexpr int XL = NS - 1;             // 64-wide steps of x in flight
  constexpr int PF = 3;                  // B operands read from LDS ahead of their products
  constexpr int PERIOD = 2 * NS;         // half steps after which slots and stages repeat (H is a multiple)
  constexpr int WAITN = lmhead_wide_wait(LEAD, XL, XB, 2);
  static_assert(WAITN < 64, "vmcnt has 6 bits");
  // separate stage arrays, so that the compiler can tell a stage being loaded
  // into LDS from the one being read (stages 4 .. 7 only with NS = 8)
  constexpr int XU8 = NS == 8 ? XU : 1;
  __shared__ __align__(16) uint4 xs0[XU][64];
  __shared__ __align__(16) uint4 xs1[XU][64];
  __shared__ __align__(16) uint4 xs2[XU][64];
  __shared__ __align__(16) uint4 xs3[XU][64];
  __shared__ __align__(16) uint4 xs4[XU8][64];
  __shared__ __align__(16) uint4 xs5[XU8][64];
  __shared__ __align__(16) uint4 xs6[XU8][64];
  __shared__ __align__(16) uint4 xs7[XU8][64];
  __shared__ WideEpi<FUSED> epi;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 15, quad = lane >> 4;
  const int K = a.K, KS = K / 64, H = 2 * KS;
  const int M = a.M;
  const int nvb = (a.V + 15) / 16;
  const int vb0 = blockIdx.x * 16 + 2 * wave;  // this wave's first 16-row vocab block (of 2)
  // buffer loads: a uniform descriptor per operand, one 32-bit vector offset per
  // lane, the step's advance in a scalar offset
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc((void*)a.w, 0, 0x7FFFFFFF, 0x00020000);
  uint32_t w_t[2];
#pragma unroll
  for (int vt = 0; vt < 2; ++vt) w_t[vt] = (uint32_t)min(vb0 + vt, nvb - 1) * (uint32_t)a.w_vb * 16u;
  const uint32_t w_ks = (uint32_t)a.w_ks * 16u;
  const uint32_t lane16 = 16u * lane;
  const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc((void*)a.x, 0, 0x7FFFFFFF, 0x00020000);
  constexpr uint32_t x_ks = XU * 1024u;  // bytes of one 64-wide step of the packed x
  // W is read once per launch: its loads carry the non-temporal hint (cache
  // policy bit 1, "nt" on gfx950) so they stream through the caches
  constexpr int kNt = 2;
  u32x4 wr[WR][2];
  auto load_w = [&](auto slot_c, int h) __attribute__((always_inline)) {
    constexpr int SL = decltype(slot_c)::value;
    h = min(h, H - 1);
    const uint32_t so = (uint32_t)(h >> 1) * w_ks + (uint32_t)(h & 1) * 1024u;
#pragma unroll
    for (int vt = 0; vt < 2; ++vt)
      wr[SL][vt] = __builtin_amdgcn_raw_buffer_load_b128(wrs, lane16, so + w_t[vt], kNt);
  };
  auto stage = [&](auto st_c) __attribute__((always_inline)) -> uint4(*)[64] {
    constexpr int ST = decltype(st_c)::value;
    if constexpr (ST < 4) {
      return ST == 0 ? xs0 : ST == 1 ? xs1 : ST == 2 ? xs2 : xs3;
    } else {
      return ST == 4 ? xs4 : ST == 5 ? xs5 : ST == 6 ? xs6 : xs7;
    }
  };
  auto load_x = [&](auto st_c, int ks) __attribute__((always_inline)) {
    uint4(*dst)[64] = stage(st_c);
    ks = min(ks, KS - 1);
#pragma unroll
    for (int i = 0; i < XB; ++i) {
      const int j = min(wave + 8 * i, XU - 1);  // operand (tile j / 2, half j % 2) of the step
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xrs, (lds_void*)&dst[j][0], 16, lane16 + 1024u * j,
                                               (uint32_t)ks * x_ks, 0, 0);
    }
  };
  f32x4 acc[2][MTP];
#pragma unroll
  for (int t = 0; t < MTP; ++t)
#pragma unroll
    for (int vt = 0; vt < 2; ++vt) acc[vt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto half = [&](auto slot_c, auto st_c, auto hf_c, int h) __attribute__((always_inline)) {
    constexpr int SL = decltype(slot_c)::value, ST = decltype(st_c)::value, HF = decltype(hf_c)::value;
    load_w(std::integral_constant<int, (SL + LEAD) % WR>{}, h + LEAD);
    if constexpr (HF == 0) load_x(std::integral_constant<int, (ST + XL) % NS>{}, (h >> 1) + XL);
    __builtin_amdgcn_sched_barrier(0);  // this half step's loads go out before its products
    uint4(*src)[64] = stage(st_c);
    bf16x8 b[PF + 1];
#pragma unroll
    for (int t = 0; t < PF; ++t) b[t] = as_bf16x8(src[2 * t + HF][lane]);
#pragma unroll
    for (int t = 0; t < MTP; ++t) {
      if (t + PF < MTP) b[(t + PF) % (PF + 1)] = as_bf16x8(src[2 * (t + PF) + HF][lane]);
#pragma unroll
      for (int vt = 0; vt < 2; ++vt)
        acc[vt][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wr[SL][vt]),
                                                              b[t % (PF + 1)], acc[vt][t], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (HF == 1) {
      wait_vmcnt<WAITN>();           // this wave's x and W of the next step have landed
      __builtin_amdgcn_s_barrier();  // and so have the other waves' x
    }
  };
  // the fused epilogue's row scales, beta, prior and query offsets: loaded first,
  // written to LDS once the prologue's loads are in flight
  float e_rho = 0.f, e_beta = 0.f, e_prior = 0.f;
  int e_qs = 0, e_row = -1;
  if constexpr (FUSED) {
    if (tid < M) e_rho = a.rho_in[tid];
    if (tid < M - a.n_queries) {  // experts: every query has one amateur row
      e_row = a.exp_seq[tid];
      e_beta = a.beta[tid];
      e_prior = a.prior[tid];
    }
    if (tid <= a.n_queries) e_qs = a.query_seq0[tid];
  }
  // prologue: the loads of half steps -LEAD .. -1 in the loop's order (half step
  // h loads W(h + LEAD) and, at even h, x(h / 2 + XL); LEAD = 2 XL + 1)
  static_assert(LEAD == 2 * XL + 1, "W and x leads");
  static_for<LEAD>([&](auto ic) __attribute__((always_inline)) {
    constexpr int h = (int)decltype(ic)::value - LEAD;
    if constexpr (h + LEAD >= 0) load_w(std::integral_constant<int, (h + LEAD) % WR>{}, h + LEAD);
    if constexpr ((h & 1) == 0 && h / 2 + XL >= 0)
      load_x(std::integral_constant<int, (h / 2 + XL) % NS>{}, h / 2 + XL);
  });
  if constexpr (FUSED) {
    if (tid < M) epi.rho[tid] = e_rho;
    if (e_row >= 0) {
      epi.beta_row[e_row] = e_beta;
      epi.prior_row[e_row] = e_prior;
    }
    if (tid <= a.n_queries) epi.qs[tid] = e_qs;
  }
  wait_vmcnt<WAITN>();
  __builtin_amdgcn_s_barrier();
  // W slot h % WR and x stage (h / 2) % NS repeat every PERIOD half steps
  for (int h = 0; h < H; h += PERIOD) {
    static_for<PERIOD>([&](auto jc) __attribute__((always_inline)) {
      constexpr int j = decltype(jc)::value;
      half(std::integral_constant<int, j % WR>{}, std::integral_constant<int, (j / 2) % NS>{},
           std::integral_constant<int, j % 2>{}, h + j);
    });
  }
  wait_vmcnt<0>();  // the loads past the end (some into LDS) have landed
  if constexpr (FUSED) {
    // Eq. 2 and the slice argmax in four passes of 64 columns through the (now
    // free) x stages. Pass p takes accumulator element p of every lane of every
    // wave: block column 32 w + 16 vt + 4 quad + p, staged as pass column
    // c = 16 (w / 2) + 4 quad + 2 (w % 2) + vt at stage c / 16, offset
    // (c % 16) RSP, rows in order. RSP = 4 (mod 32): a wave's stores hit each
    // bank twice, and 16-byte reads of one row in eight consecutive columns
    // fall in distinct banks; RSP >= M + kWideOverRead, so reads of whole 4-row
    // groups past a query's last row stay in the column. Each query has T
    // threads (a power of two); a thread takes 64 / T columns, or with T > 64
    // es = T / 64 adjacent threads share a column and split its 4-row groups,
    // merging (score, expert) with the lower expert on equal scores (the
    // sequential scan's choice). After the last pass the query's threads merge
    // their best two tokens (shuffles, then LDS across waves) into the block's
    // first fuse_part slot; its second slot (if any) gets an empty candidate.
    constexpr int NCP = 64;
    static_assert(16 * (16 * MTP + kWideOverRead + 35) <= XU * 64 * 4, "16 padded columns per stage");
    const int RSP = (((M + kWideOverRead + 27) >> 5) << 5) + 4;
    auto colp = [&](int c) -> float* {
      const int q = c >> 4;
      float* base = q == 0 ? (float*)&xs0[0][0] : q == 1 ? (float*)&xs1[0][0] : q == 2 ? (float*)&xs2[0][0]
                                                                                   : (float*)&xs3[0][0];
      return base + (c & 15) * RSP;
    };
    int T = 512;
    while (T > 2 && T * a.n_queries > 512) T >>= 1;
    const int es = T > 64 ? T / 64 : 1, cpl = T < 64 ? 64 / T : 1;
    const int qb = tid / T, ti = tid % T, sp = ti % es;
    const bool active = qb < a.n_queries;
    const int s0 = active ? epi.qs[qb] : 0;
    const int N = active ? epi.qs[qb + 1] - s0 - 1 : 0;
    const int rb = (s0 + 1) & ~3, nb = ((s0 + N) >> 2) - (rb >> 2) + 1;  // 4-row groups holding the experts
    __shared__ Top2 red[8];
    Top2 cand{kNegInf, 0x7FFFFFFF, 0, kNegInf, 0x7FFFFFFF};
    __syncthreads();  // every wave is done with the x stages
#pragma unroll 1
    for (int p = 0; p < 4; ++p) {
#pragma unroll
      for (int t = 0; t < MTP; ++t) {
        const int m = 16 * t + col;
        if (m >= M) continue;
        const float rho = epi.rho[m];
#pragma unroll
        for (int vt = 0; vt < 2; ++vt) {
          const f32x4 cc = acc[vt][t];
          const float x = p == 0 ? cc[0] : p == 1 ? cc[1] : p == 2 ? cc[2] : cc[3];
          colp(16 * (wave >> 1) + 4 * quad + 2 * (wave & 1) + vt)[m] = x * rho;
        }
      }
      __syncthreads();
      if (active) {
        for (int i = 0; i < cpl; ++i) {
          const int c = es > 1 ? ti / es : ti + T * i;
          const int wc = 2 * (c >> 4) + ((c >> 1) & 1);
          const int v = blockIdx.x * 256 + 32 * wc + 16 * (c & 1) + 4 * ((c >> 2) & 3) + p;
          const float* cp = colp(c);
          float best = kNegInf;
          int bk = 0;
          if (v < a.V) {
            const float sa = cp[s0];
            for (int ib = sp; ib < nb; ib += 2 * es) {
              const int r1 = rb + 4 * ib, r2 = r1 + 4 * es;
              const float4 x1 = *(const float4*)(cp + r1), x2 = *(const float4*)(cp + r2);
              const float4 b1 = *(const float4*)(epi.beta_row + r1), b2 = *(const float4*)(epi.beta_row + r2);
              const float4 p1 = *(const float4*)(epi.prior_row + r1), p2 = *(const float4*)(epi.prior_row + r2);
              eq2_rows4(x1, b1, p1, sa, r1 - s0, N, best, bk);
              eq2_rows4(x2, b2, p2, sa, r2 - s0, N, best, bk);
            }
          }
          for (int o = 1; o < es; o <<= 1) {
            const float ob = __shfl_xor(best, o);
            const int ok = __shfl_xor(bk, o);
            if (ob > best || (ob == best && ok < bk)) {
              best = ob;
              bk = ok;
            }
          }
          if (sp == 0 && v < a.V) cand = merge(cand, Top2{best, v, bk, kNegInf, 0x7FFFFFFF});
        }
      }
      __syncthreads();  // before the next pass writes the stages
    }
    // the query's best two tokens over the block's 256 columns
    for (int o = min(T, 64) >> 1; o >= 1; o >>= 1) cand = merge(cand, shfl_top2(cand, o));
    if (T > 64) {
      if (lane == 0) red[wave] = cand;
      __syncthreads();
      if (ti == 0)
        for (int w = 1; w < T / 64; ++w) cand = merge(cand, red[wave + w]);
    }
    if (ti == 0 && active) {
      float* pp = a.fuse_part + ((size_t)qb * a.fuse_nblk + 2 * blockIdx.x) * 5;
      pp[0] = cand.v1; pp[1] = __int_as_float(cand.i1); pp[2] = __int_as_float(cand.k1);
      pp[3] = cand.v2; pp[4] = __int_as_float(cand.i2);
      if (2 * (int)blockIdx.x + 1 < a.fuse_nblk) {  // (the last block's second slot may not exist)
        pp[5] = kNegInf; pp[6] = __int_as_float(0x7FFFFFFF); pp[7] = __int_as_float(0);
        pp[8] = kNegInf; pp[9] = __int_as_float(0x7FFFFFFF);
      }
    }
    return;
  }
#pragma unroll
  for (int t = 0; t < MTP; ++t) {
    const int m = 16 * t + col;
    if (m >= M) continue;
    const float rho = a.rho_in[m];
#pragma unroll
    for (int vt = 0; vt < 2; ++vt) {
      if (vb0 + vt >= nvb) continue;
      const int v = 16 * (vb0 + vt) + 4 * quad;
      float* out = a.logits + (size_t)m * a.V + v;
      const f32x4 cc = acc[vt][t];
      if (v + 3 < a.V && (a.V & 3) == 0) {
        *(float4*)out = make_float4(cc[0] * rho, cc[1] * rho, cc[2] * rho, cc[3] * rho);
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (v + r < a.V) out[r] = cc[r] * rho;
      }
    }
  }
}

// fp32 LM head for small validation shapes: one thread per vocab row.
__global__ __launch_bounds__(256) void k_lmhead_f32(LmArgs a) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= a.V) return;
  const float* W = (const float*)a.w + (size_t)v * a.K;
  for (int m = 0; m < a.M; ++m) {
    const float* x = (const float*)a.x + (size_t)m * a.K;
    float ss = 0.f, dot = 0.f;
    for (int k = 0; k < a.K; ++k) {
      ss += x[k] * x[k];
      dot += x[k] * W[k];
    }
    const float rho = a.rms ? 1.0f / sqrtf(ss / (float)a.K + 1e-5f) : 1.0f;
    a.logits[(size_t)m * a.V + v] = dot * rho;
  }
}

// ---------------------------------------------------------- Eq. 2 and Eq. 3

// Eq. 2 and the best two tokens of one SW-token vocabulary slice per block
// (SW = 1024, or 512 when 1024-token slices would leave compute units idle).
// Per token v:
//   s_hat_k(v) = ((1 + beta_k) s_k(v) - beta_k s_0(v)) + gamma ln r_k     (Eq. 2)
// evaluated in float32 in exactly that order without fused multiply-adds,
// S(v) = max over experts 1..N (lowest k on ties). A block of 4 waves owns
// SW consecutive tokens; wave w takes the experts of its quarter of 1..N and
// reads their rows in 4 SW-byte runs: lane l holds tokens 4l + 256i .. +3 (i < SW/256),
// one 16-byte load each (VEC: rows 16-byte aligned, V % 4 == 0; otherwise
// 4-byte loads), so every wave load is a contiguous 1 KiB of a row and a batch
// of NB rows keeps 4 NB loads in flight before any arithmetic (rows past the
// quarter re-read its last row and are masked by selects). The waves' per-token
// maxima meet in LDS and are combined in wave order (ties keep the lower k),
// then each wave takes 256 of the tokens, the lanes' candidates are merged by
// shuffles and the waves' by LDS; the slice's best two tokens go to
// part[b][slice] for k_fuse_final. (A single launch, the last block merging the
// slices behind an agent-scope release/acquire counter, measured 2x slower at
// one query and 7x at sixteen: the release writes back the L2 of every wave's
// compute unit.)
template <bool VEC>
__device__ __forceinline__ float4 load_tok4(const float* row, int v0, int V) {
  if constexpr (VEC) {
    return *(const float4*)(row + min(v0, V - 4));
  } else {
    return make_float4(row[min(v0, V - 1)], row[min(v0 + 1, V - 1)], row[min(v0 + 2, V - 1)],
                       row[min(v0 + 3, V - 1)]);
  }
}

__device__ __forceinline__ void fuse_write_outputs(const FuseArgs& a, int b, const Top2& r) {
  a.tokens_out[(size_t)b * a.tok_stride] = r.i1;
  a.prev_tok[b] = r.i1;
  if (a.winner) a.winner[b] = r.k1;
  if (a.top1) a.top1[b] = r.v1;
  if (a.top2) a.top2[b] = r.v2;
}

__device__ __forceinline__ Top2 wave_top2(Top2 c) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) c = merge(c, shfl_top2(c, o));
  return c;
}

template <bool VEC, int NB, int SW>
__global__ __launch_bounds__(256) void k_fuse(FuseArgs a) {
#pragma clang fp contract(off)
  constexpr int RI = SW / 256;  // 16-byte loads per lane and row
  __shared__ float sbest[4][SW];
  __shared__ int sk[4][SW];
  __shared__ Top2 swave[4];
  const int b = blockIdx.y, lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // the first queries' row offsets travel in the kernel arguments (no dependent load)
  const bool inl = b < kFuseInlineQueries;
  const int s0 = inl ? a.inl_seq0[b] : a.query_seq0[b];
  const int N = (inl ? a.inl_seq0[b + 1] : a.query_seq0[b + 1]) - s0 - 1;
  const int e0 = inl ? a.inl_exp0[b] : a.query_exp0[b];
  const int per = (N + 3) / 4;                       // experts per wave
  const int k_lo = 1 + wave * per, k_hi = min(N, k_lo + per - 1);
  const int vb = blockIdx.x * SW;
  const float* L0 = a.logits + (size_t)s0 * a.V;
  float sa[4 * RI], best[4 * RI];
  int bk[4 * RI];
#pragma unroll
  for (int i = 0; i < RI; ++i) {
    const float4 t = load_tok4<VEC>(L0, vb + 256 * i + 4 * lane, a.V);
    sa[4 * i] = t.x; sa[4 * i + 1] = t.y; sa[4 * i + 2] = t.z; sa[4 * i + 3] = t.w;
  }
#pragma unroll
  for (int u = 0; u < 4 * RI; ++u) { best[u] = kNegInf; bk[u] = 0; }
  for (int kb = k_lo; kb <= k_hi; kb += NB) {
    float4 x[NB][RI];
    float cb[NB], cp[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const float* row = L0 + (size_t)min(kb + j, k_hi) * a.V;
#pragma unroll
      for (int i = 0; i < RI; ++i) x[j][i] = load_tok4<VEC>(row, vb + 256 * i + 4 * lane, a.V);
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int e = e0 + min(kb + j, k_hi) - 1;
      cb[j] = a.beta[e];
      cp[j] = a.prior[e];
    }
    __builtin_amdgcn_sched_barrier(0);  // all of the batch's loads go out before the arithmetic
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int k = kb + j;
      const bool ok = k <= k_hi;
      const float beta = cb[j], pr = cp[j];
      const float coef = 1.0f + beta;
#pragma unroll
      for (int i = 0; i < RI; ++i) {
        const float xs[4] = {x[j][i].x, x[j][i].y, x[j][i].z, x[j][i].w};
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int u = 4 * i + c;
          const float t1 = coef * xs[c];
          const float t2 = beta * sa[u];
          const float val = (t1 - t2) + pr;
          const bool up = ok && val > best[u];
          best[u] = up ? val : best[u];
          bk[u] = up ? k : bk[u];
        }
      }
    }
  }
  // per-token maxima of the four expert ranges, combined in wave order
#pragma unroll
  for (int i = 0; i < RI; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      sbest[wave][256 * i + 4 * lane + c] = best[4 * i + c];
      sk[wave][256 * i + 4 * lane + c] = bk[4 * i + c];
    }
  __syncthreads();
  Top2 cand{kNegInf, 0x7FFFFFFF, 0, kNegInf, 0x7FFFFFFF};
#pragma unroll
  for (int c = 0; c < SW / 256; ++c) {  // wave w finishes tokens w SW/4 .. (w + 1) SW/4 - 1
    const int t = SW / 4 * wave + (SW / 256) * lane + c;
    float v = sbest[0][t];
    int k = sk[0][t];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      const float vw = sbest[w][t];
      if (vw > v) { v = vw; k = sk[w][t]; }
    }
    if (vb + t < a.V) cand = merge(cand, Top2{v, vb + t, k, kNegInf, 0x7FFFFFFF});
  }
  cand = wave_top2(cand);
  if (lane == 0) swave[wave] = cand;
  __syncthreads();
  if (threadIdx.x == 0) {
    Top2 r = swave[0];
#pragma unroll
    for (int w = 1; w < 4; ++w) r = merge(r, swave[w]);
    float* p = a.part + ((size_t)b * a.nblk + blockIdx.x) * 5;
    p[0] = r.v1; p[1] = __int_as_float(r.i1); p[2] = __int_as_float(r.k1);
    p[3] = r.v2; p[4] = __int_as_float(r.i2);
  }
}

// One block per query: merges the vocabulary slices' candidates and writes
// y_t (Eq. 3), the expert that scored it, and the two best distinct scores.
__global__ __launch_bounds__(kFuseBlock) void k_fuse_final(FuseArgs a) {
  const int b = blockIdx.x;
  Top2 r{kNegInf, 0x7FFFFFFF, 0, kNegInf, 0x7FFFFFFF};
  for (int i = threadIdx.x; i < a.nblk; i += blockDim.x) {
    const float* p = a.part + ((size_t)b * a.nblk + i) * 5;
    Top2 x{p[0], __float_as_int(p[1]), __float_as_int(p[2]), p[3], __float_as_int(p[4])};
    r = merge(r, x);
  }
  r = block_top2<kFuseBlock / 64>(r);
  if (threadIdx.x == 0) fuse_write_outputs(a, b, r);
}

// ---------------------------------------------------------------- dynamic beta

__device__ float block_reduce_max(float v) {
  __shared__ float red[4];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  const float r = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  return r;
}

__device__ float block_reduce_sum(float v) {
  __shared__ float red[4];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  const float r = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return r;
}

constexpr float kLog2E = 1.44269504088896341f;
static_assert(kBetaChunk % 1024 == 0, "whole 16-byte loads per thread");

// A thread's kBetaChunk / 256 values of a chunk [v0, v1) of a logits row, in
// registers (16-byte loads when rows are 16-byte aligned); -inf past v1.
__device__ __forceinline__ void beta_chunk_values(const float* row, int V, int v0, int v1,
                                                  float (&x)[kBetaChunk / 256]) {
  constexpr int PER = kBetaChunk / 256;
  if ((V & 3) == 0) {
#pragma unroll
    for (int i = 0; i < PER / 4; ++i) {
      const int v = v0 + 4 * (threadIdx.x + 256 * i);
      float4 t = make_float4(kNegInf, kNegInf, kNegInf, kNegInf);
      if (v < v1) t = *(const float4*)(row + v);
      x[4 * i] = t.x; x[4 * i + 1] = t.y; x[4 * i + 2] = t.z; x[4 * i + 3] = t.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int v = v0 + threadIdx.x + 256 * i;
      x[i] = v < v1 ? row[v] : kNegInf;
    }
  }
}

// Per (row, vocab chunk): chunk max M_c and sum 2^((s - M_c) log2 e), in one
// pass (the block's values stay in registers between the two reductions).
__global__ __launch_bounds__(256) void k_beta_lse(BetaArgs a) {
  constexpr int PER = kBetaChunk / 256;
  const int s = blockIdx.y, ch = blockIdx.x;
  const int v0 = ch * kBetaChunk, v1 = min(a.V, v0 + kBetaChunk);
  float x[PER];
  beta_chunk_values(a.logits + (size_t)s * a.V, a.V, v0, v1, x);
  float m = kNegInf;
#pragma unroll
  for (int i = 0; i < PER; ++i) m = fmaxf(m, x[i]);
  m = block_reduce_max(m);
  float sum = 0.f;
#pragma unroll
  for (int i = 0; i < PER; ++i) sum += x[i] == kNegInf ? 0.f : __builtin_amdgcn_exp2f((x[i] - m) * kLog2E);
  sum = block_reduce_sum(sum);
  if (threadIdx.x == 0) {
    a.lse_part[((size_t)s * a.nchunk + ch) * 2] = m;
    a.lse_part[((size_t)s * a.nchunk + ch) * 2 + 1] = sum;
  }
}

// Base-2 log-sum-exp of a row from its chunk partials, by one wave (lanes over
// chunks, then shuffles); every lane returns it.
__device__ __forceinline__ float wave_row_lse2(const BetaArgs& a, int s) {
  const float* p = a.lse_part + (size_t)s * a.nchunk * 2;
  const int lane = threadIdx.x & 63;
  float m = kNegInf;
  for (int c = lane; c < a.nchunk; c += 64) m = fmaxf(m, p[2 * c]);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
  float sum = 0.f;
  for (int c = lane; c < a.nchunk; c += 64) sum += p[2 * c + 1] * __builtin_amdgcn_exp2f((p[2 * c] - m) * kLog2E);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) sum += __shfl_xor(sum, o);
  return m * kLog2E + __builtin_amdgcn_logf(sum);
}

// beta_k = JSD(p_k || p_0) in bits (first step, dynamic mode; Section 3 reads
// beta from AdaCAD's with-context vs no-context divergence). Per (expert,
// chunk) partial sums. With base-2 log-probabilities lp, lq, d = lp - lq,
// hi = max(lp, lq), t = 2^-|d| and g = log2(1 + t), the mixture m = (p + q) / 2
// has log2 m = hi + g - 1, so the larger probability 2^hi contributes
// 2^hi (1 - g) / 2 and the smaller 2^hi t (1 - |d| - g) / 2: no difference of
// two large logarithms is formed.
__global__ __launch_bounds__(256) void k_beta_jsd(BetaArgs a) {
  constexpr int PER = kBetaChunk / 256;
  const int e = blockIdx.y, ch = blockIdx.x;
  const int sk = a.exp_seq[e];
  const int s0 = a.query_seq0[a.exp_query[e]];
  const int v0 = ch * kBetaChunk, v1 = min(a.V, v0 + kBetaChunk);
  float xk[PER], x0[PER];
  beta_chunk_values(a.logits + (size_t)sk * a.V, a.V, v0, v1, xk);
  beta_chunk_values(a.logits + (size_t)s0 * a.V, a.V, v0, v1, x0);
  __shared__ float lse2[2];
  if (threadIdx.x < 64) {
    const float lk = wave_row_lse2(a, sk), l0 = wave_row_lse2(a, s0);
    if (threadIdx.x == 0) {
      lse2[0] = lk;
      lse2[1] = l0;
    }
  }
  __syncthreads();
  const float lk = lse2[0], l0 = lse2[1];
  float acc = 0.f;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    if (x0[i] == kNegInf) continue;  // past the chunk's end
    const float lp = xk[i] * kLog2E - lk, lq = x0[i] * kLog2E - l0;
    const float ad = fabsf(lp - lq), hi = fmaxf(lp, lq);
    const float t = __builtin_amdgcn_exp2f(-ad);
    const float g = __builtin_amdgcn_logf(1.0f + t);
    acc += 0.5f * __builtin_amdgcn_exp2f(hi) * ((1.0f - g) + t * ((1.0f - ad) - g));
  }
  acc = block_reduce_sum(acc);
  if (threadIdx.x == 0) a.jsd_part[(size_t)e * a.nchunk + ch] = acc;
}

// beta_k = sum of expert k's chunk partials (bits): one wave per expert.
__global__ __launch_bounds__(64) void k_beta_final(BetaArgs a, int n_exp) {
  const int e = blockIdx.x;
  if (e >= n_exp) return;
  float tot = 0.f;
  for (int c = threadIdx.x; c < a.nchunk; c += 64) tot += a.jsd_part[(size_t)e * a.nchunk + c];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) tot += __shfl_xor(tot, o);
  if (threadIdx.x == 0) a.beta[e] = tot;
}

// Scalar beta (one per query): the mean of the query's per-expert divergences,
// summed in expert order, written back to every expert of the query.
__global__ __launch_bounds__(64) void k_beta_mean(BetaArgs a) {
  const int b = blockIdx.x;
  const int e0 = a.query_exp0[b], e1 = a.query_exp0[b + 1];
  if (threadIdx.x == 0) {
    float tot = 0.f;
    for (int e = e0; e < e1; ++e) tot += a.beta[e];
    const float m = tot / (float)(e1 - e0);
    for (int e = e0; e < e1; ++e) a.beta[e] = m;
  }
}

// ------------------------------------------------ MoE / PoE aggregation

// Per (expert, vocabulary chunk): max and sum of exp(c - max) of the contrastive
// logits c = (1 + beta) s_k - beta s_0 (Eq. 2's order, no contraction).
__global__ __launch_bounds__(256) void k_agg_lse(AggArgs a) {
#pragma clang fp contract(off)
  const int e = blockIdx.y, ch = blockIdx.x;
  const float* rk = a.logits + (size_t)a.exp_seq[e] * a.V;
  const float* r0 = a.logits + (size_t)a.query_seq0[a.exp_query[e]] * a.V;
  const float beta = a.beta[e], coef = 1.0f + beta;
  const int v0 = ch * kBetaChunk, v1 = min(a.V, v0 + kBetaChunk);
  auto cval = [&](int v) { const float t1 = coef * rk[v]; const float t2 = beta * r0[v]; return t1 - t2; };
  float m = kNegInf;
  for (int v = v0 + threadIdx.x; v < v1; v += blockDim.x) m = fmaxf(m, cval(v));
  m = block_reduce_max(m);
  float sum = 0.f;
  for (int v = v0 + threadIdx.x; v < v1; v += blockDim.x) sum += expf(cval(v) - m);
  sum = block_reduce_sum(sum);
  if (threadIdx.x == 0) {
    a.lse_part[((size_t)e * a.nchunk + ch) * 2] = m;
    a.lse_part[((size_t)e * a.nchunk + ch) * 2 + 1] = sum;
  }
}

// lse_k from the chunk partials, in chunk order.
__global__ __launch_bounds__(256) void k_agg_lse_final(AggArgs a, int n_exp) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= n_exp) return;
  const float* p = a.lse_part + (size_t)e * a.nchunk * 2;
  float m = kNegInf;
  for (int c = 0; c < a.nchunk; ++c) m = fmaxf(m, p[2 * c]);
  float sum = 0.f;
  for (int c = 0; c < a.nchunk; ++c) sum += p[2 * c + 1] * expf(p[2 * c] - m);
  a.lse[e] = m + logf(sum);
}

// One block per (query, 256-token slice): per token v the experts' weighted
// log-probabilities j_k = log pi_k + c_k(v) - lse_k, then
//   MoE: log sum_k exp(j_k)  (running max and rescaled sum, expert order)
//   PoE: sum_k pi_k (c_k(v) - lse_k)
// and the expert with the largest j_k (lowest k on ties); the block's best two
// tokens go to the same partial buffer k_fuse_final merges.
__global__ __launch_bounds__(kFuseBlock) void k_agg(AggArgs a) {
#pragma clang fp contract(off)
  const int b = blockIdx.y;
  const int s0 = a.query_seq0[b];
  const int N = a.query_seq0[b + 1] - s0 - 1;
  const int e0 = a.query_exp0[b];
  const int v = blockIdx.x * kFuseBlock + threadIdx.x;
  Top2 c{kNegInf, 0x7FFFFFFF, 0, kNegInf, 0x7FFFFFFF};
  if (v < a.V) {
    const float sa = a.logits[(size_t)s0 * a.V + v];
    float m = kNegInf, sum = 0.f, prod = 0.f, jbest = kNegInf;
    int bk = 0;
    for (int k = 1; k <= N; ++k) {
      const int e = e0 + k - 1;
      const float beta = a.beta[e], coef = 1.0f + beta;
      const float t1 = coef * a.logits[(size_t)(s0 + k) * a.V + v];
      const float t2 = beta * sa;
      const float lp = (t1 - t2) - a.lse[e];
      const float j = a.logw[e] + lp;
      if (j > jbest) { jbest = j; bk = k; }
      if (a.product) {
        prod += expf(a.logw[e]) * lp;
      } else if (j > m) {
        sum = sum * expf(m - j) + 1.0f;
        m = j;
      } else {
        sum += expf(j - m);
      }
    }
    c.v1 = a.product ? prod : m + logf(sum);
    c.i1 = v;
    c.k1 = bk;
  }
  c = block_top2<kFuseBlock / 64>(c);
  if (threadIdx.x == 0) {
    float* p = a.part + ((size_t)b * a.nblk + blockIdx.x) * 5;
    p[0] = c.v1; p[1] = __int_as_float(c.i1); p[2] = __int_as_float(c.k1);
    p[3] = c.v2; p[4] = __int_as_float(c.i2);
  }
}

// --------------------------------------------------- generation input synth

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;
__device__ __forceinline__ uint64_t fold(uint64_t k, uint64_t f) { return mix64((k ^ f) + kGolden); }

template <bool BF16>
__device__ void synth_fill(void* dst, size_t off, uint64_t key, int n, float scale) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const uint64_t h = mix64(key + (uint64_t)(i + 1) * kGolden);
    const int u = (int)(h & 0xFFFF) + (int)((h >> 16) & 0xFFFF) + (int)((h >> 32) & 0xFFFF) + (int)(h >> 48);
    const float v = (float)(u - 131070) * scale;
    if (BF16) ((uint16_t*)dst)[off + i] = (uint16_t)f2bf(v);
    else ((float*)dst)[off + i] = v;
  }
}

// Step-t inputs of sequence s, layer l from the previous token of its query:
// q = stream(fold(seed, 0x51, t, s, l, y)), k_new with tag 0x4B, v_new with 0x56.
template <bool BF16>
__global__ __launch_bounds__(256) void k_synth(SynthArgs a) {
  const int s = blockIdx.x / a.n_layers, l = blockIdx.x % a.n_layers;
  const int y = a.use_first ? a.first_token : a.prev_tok[a.seq_query[s]];
  uint64_t base[3];
  const uint64_t tags[3] = {0x51, 0x4B, 0x56};
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    uint64_t k = fold(a.seed, tags[i]);
    k = fold(k, (uint64_t)a.t);
    k = fold(k, (uint64_t)s);
    k = fold(k, (uint64_t)l);
    base[i] = fold(k, (uint64_t)y);
  }
  const size_t row = (size_t)s * a.n_layers + l;
  synth_fill<BF16>(a.q, row * a.qdim, base[0], a.qdim, a.value_scale);
  synth_fill<BF16>(a.k_new, row * a.kvdim, base[1], a.kvdim, a.value_scale);
  synth_fill<BF16>(a.v_new, row * a.kvdim, base[2], a.kvdim, a.value_scale);
}

// ------------------------------------------------------------ decoder stack

constexpr int kProjWaves = 8;  // waves per projection block


// Decoder projection for the rows of one decode step (M <= 16 NT <= 48 rows,
// in the matrix cores' N dimension): K-slice partial sums part[split][m][n] = sum_{k in slice}
// x[m][k] W[n][k] on the matrix cores, C^T[16 columns x 16 rows] += W[16 x 32]
// X^T[32 x 16] (v_mfma_f32_16x16x32_bf16); k_proj_reduce adds the slices in
// order and applies the projection's epilogue.
// Block b covers column group b / ksplit (8 TPW consecutive 16-column tiles,
// TPW per wave) over K slice b % ksplit. The block first stages its x slice
// (rows x slice, row-major, rows padded by 16 bytes against bank conflicts) in
// LDS with coalesced loads; each wave then streams only its packed W tiles
// (contiguous 1 KiB loads, every byte read once) through an R-deep register ring
// and reads its x operands from LDS, so the whole register ring holds W bytes
// in flight. The barrier after staging waits on LDS only; it does not drain the
// ring.
template <int NT, int TPW>
__global__ __launch_bounds__(64 * kProjWaves) void k_proj(GemmArgs a) {
  constexpr int WPB = kProjWaves, CT = WPB * TPW, R = TPW == 1 ? 8 : 5;
  extern __shared__ __align__(16) uint16_t xs[];
  // the wave index (and so the tiles) is scalar; the ring's tail guards depend
  // only on kernel arguments, so they are branches: matrix-core instructions do
  // not honour EXEC, a guard turned into an EXEC mask would not stop them
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15, quad = lane >> 4;
  const int grp = blockIdx.x / a.ksplit, split = blockIdx.x - grp * a.ksplit;
  const int K = a.K, KS = K / 64;
  const int ks0 = split * KS / a.ksplit;
  const int n = (split + 1) * KS / a.ksplit - ks0;
  const int LDX = 64 * n + 8;  // staged row length (elements)
  const int N = 16 * a.n_tiles;
  // packed W: tile (t, ks) at (t * t_vb + ks * t_ks) * 128 16-byte units
  const size_t t_vb = kProjKMajor ? 1 : KS, t_ks = kProjKMajor ? (size_t)a.n_tiles : 1;
  const uint4* wt[TPW];
#pragma unroll
  for (int tt = 0; tt < TPW; ++tt)
    wt[tt] = (const uint4*)a.w + ((size_t)min(grp * CT + wave * TPW + tt, a.n_tiles - 1) * t_vb + ks0 * t_ks) * 128 +
             lane;

  const int m0 = 0, rows = a.M;  // one row group: M <= 16 NT
  f32x4 acc[TPW][NT];
#pragma unroll
  for (int tt = 0; tt < TPW; ++tt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[tt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  struct Stage { uint4 w[TPW][2]; };
  Stage st[R];
  auto load = [&](Stage& S, int i) __attribute__((always_inline)) {
    i = min(i, n - 1);  // past the end: the last step again (a cache hit), the ring stays branch-free
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      S.w[tt][0] = ld_w<true>(&wt[tt][(size_t)i * t_ks * 128]);
      S.w[tt][1] = ld_w<true>(&wt[tt][(size_t)i * t_ks * 128 + 64]);
    }
  };
  // x operand rows of this lane in LDS (rows past the group's end read the last row)
  const uint16_t* xl[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) xl[nt] = xs + (size_t)min(16 * nt + col, rows - 1) * LDX + 16 * quad;
  auto mma = [&](const Stage& S, int i) __attribute__((always_inline)) {
    uint4 xv[NT][2];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      xv[nt][0] = *(const uint4*)(xl[nt] + 64 * i);
      xv[nt][1] = *(const uint4*)(xl[nt] + 64 * i + 8);
    }
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        acc[tt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(S.w[tt][0]), as_bf16x8(xv[nt][0]),
                                                              acc[tt][nt], 0, 0, 0);
        acc[tt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(S.w[tt][1]), as_bf16x8(xv[nt][1]),
                                                              acc[tt][nt], 0, 0, 0);
      }
  };
  // Stage the x slice: units of 8 elements, consecutive threads along a row, SB
  // units per thread in flight at once (indices past the end repeat the last
  // unit: same value, same place). The first batch is issued before the W ring,
  // so its wait leaves the ring in flight; a load-then-store loop paid one
  // memory round trip per unit with the ring stalled.
  constexpr int SB = 8;
  const int upr = 8 * n, units = rows * upr;  // units per row, in all
  uint4 xv[SB];
  int xo[SB];  // LDS element offsets of the batch's units
#pragma unroll
  for (int j = 0; j < SB; ++j) {
    const int u = min((int)threadIdx.x + j * 64 * WPB, units - 1), r = u / upr, c = u - r * upr;
    xv[j] = *(const uint4*)(a.x + (size_t)(m0 + r) * K + 64 * ks0 + 8 * c);
    xo[j] = r * LDX + 8 * c;
  }
#pragma unroll
  for (int j = 0; j < R; ++j) load(st[j], j);
#pragma unroll
  for (int j = 0; j < SB; ++j) *(uint4*)(xs + xo[j]) = xv[j];
  for (int u0 = threadIdx.x + SB * 64 * WPB; u0 < units; u0 += SB * 64 * WPB) {
#pragma unroll
    for (int j = 0; j < SB; ++j) {
      const int u = min(u0 + j * 64 * WPB, units - 1), r = u / upr, c = u - r * upr;
      xv[j] = *(const uint4*)(a.x + (size_t)(m0 + r) * K + 64 * ks0 + 8 * c);
      xo[j] = r * LDX + 8 * c;
    }
#pragma unroll
    for (int j = 0; j < SB; ++j) *(uint4*)(xs + xo[j]) = xv[j];
  }
  __syncthreads();
  for (int i = 0; i < n; i += R) {
#pragma unroll
    for (int j = 0; j < R; ++j) {
      if (i + j < n) mma(st[j], i + j);
      load(st[j], i + j + R);
    }
  }
#pragma unroll
  for (int tt = 0; tt < TPW; ++tt) {
    const int tile = grp * CT + wave * TPW + tt;
    if (tile < a.n_tiles) {
      float* dst = a.part + (size_t)split * a.M * N + 16 * tile + 4 * quad;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int m = m0 + 16 * nt + col;
        if (m < a.M)
          *(float4*)(dst + (size_t)m * N) = make_float4(acc[tt][nt][0], acc[tt][nt][1], acc[tt][nt][2], acc[tt][nt][3]);
      }
    }
  }
}

// Sum of a projection's K-slice partials (in slice order: deterministic), then
// its epilogue. Block (x, y): row m = y, 4-column output groups 256 x .. 256 x + 255.
//   kEpiQkv    row scale from the norm's sums of squares; RoPE on q and k
//              (pairs (2i, 2i+1) at the sequence's position); q to the
//              attention's query buffer, k and v into the paged cache;
//   kEpiResid  h += out, then the next norm's input bf16(h * g) and the
//              per-16-column sums of h^2 its row scale is built from;
//   kEpiSwiglu packed tiles alternate gate / up (16 columns each): with the row
//              scale, act = bf16(silu(gate) * up) for the F MLP columns.
// KMAX >= ksplit: every slice's load is issued before any is used (slots past
// ksplit re-read the last slice, so the count is fixed and branch-free), then
// the slices are added in order; a runtime loop of load-then-add paid one
// memory round trip per slice.
template <int EPI, int KMAX>
__global__ __launch_bounds__(256) void k_proj_reduce(GemmArgs a) {
  const int m = blockIdx.y, N = 16 * a.n_tiles;
  const int c4 = blockIdx.x * 256 + threadIdx.x;
  const int n0 = 4 * c4;
  const int ncols = EPI == kEpiSwiglu ? N / 2 : N;
  const bool valid = n0 < ncols;
  const int nc = valid ? n0 : ncols - 4;  // in-range column for the loads of threads past the end
  const int last = a.ksplit - 1;
  auto slice = [&](int sp) __attribute__((always_inline)) {
    return a.part + ((size_t)min(sp, last) * a.M + m) * N;
  };
  float4 pv[KMAX], uv[EPI == kEpiSwiglu ? KMAX : 1];
  if constexpr (EPI == kEpiSwiglu) {
    const int ng = 32 * (nc / 16) + nc % 16;  // gate column in the interleaved tiles; up is 16 further
#pragma unroll
    for (int sp = 0; sp < KMAX; ++sp) {
      pv[sp] = *(const float4*)(slice(sp) + ng);
      uv[sp] = *(const float4*)(slice(sp) + ng + 16);
    }
  } else {
#pragma unroll
    for (int sp = 0; sp < KMAX; ++sp) pv[sp] = *(const float4*)(slice(sp) + nc);
  }
  // the epilogue's own inputs, in the same round trip: the residual row and the
  // next norm's weights, or the row's position and the page of its new K/V row
  float4 h_in = make_float4(0.f, 0.f, 0.f, 0.f);
  uint2 g_in = make_uint2(0u, 0u);
  int pos = 0, phys = 0;
  float4 rope = make_float4(1.f, 0.f, 1.f, 0.f);
  if constexpr (EPI == kEpiResid) {
    h_in = *(const float4*)(a.h + (size_t)m * N + nc);  // residual row stride: hidden = N
    g_in = *(const uint2*)(a.g_next + nc);
  } else if constexpr (EPI == kEpiQkv) {
    pos = a.len0[m] + a.t;
    phys = a.page_table[(size_t)m * a.maxpps + pos / kPage];
    // (cos, sin) of the pairs (nc % D) / 2 and + 1 (q and k sections start at multiples of D)
    rope = *(const float4*)(a.rope + (size_t)pos * (a.head_dim / 2) + (nc % a.head_dim) / 2);
  }
  float rho = 1.0f;
  if (EPI != kEpiResid && a.rho_in) {
    rho = a.rho_in[m];
  } else if (EPI != kEpiResid && a.ss_in) {
    float t = 0.f;
    for (int p = threadIdx.x; p < a.ss_parts; p += 256) t += a.ss_in[(size_t)m * a.ld_ss + p];
    rho = 1.0f / sqrtf(block_reduce_sum(t) * a.inv_norm_dim + a.eps);
  }
  if constexpr (EPI == kEpiSwiglu) {
    if (!valid) return;
    float g[4] = {0.f, 0.f, 0.f, 0.f}, u[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int sp = 0; sp < KMAX; ++sp) {
      if (sp < a.ksplit) {
        const float4 gv = pv[sp], u4 = uv[sp];
        g[0] += gv.x; g[1] += gv.y; g[2] += gv.z; g[3] += gv.w;
        u[0] += u4.x; u[1] += u4.y; u[2] += u4.z; u[3] += u4.w;
      }
    }
    uint32_t o[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float gg = g[q] * rho, uu = u[q] * rho;
      o[q] = f2bf(gg / (1.0f + expf(-gg)) * uu);
    }
    *(uint2*)(a.act + (size_t)m * a.F + n0) = make_uint2(o[0] | (o[1] << 16), o[2] | (o[3] << 16));
    return;
  }
  float o[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int sp = 0; sp < KMAX; ++sp) {
    if (sp < a.ksplit) {
      const float4 v = pv[sp];
      o[0] += v.x;
      o[1] += v.y;
      o[2] += v.z;
      o[3] += v.w;
    }
  }
  if constexpr (EPI == kEpiResid) {
    float ss = 0.f;
    if (valid) {
      float* hp = a.h + (size_t)m * N + n0;
      float4 hv = h_in;
      hv.x += o[0];
      hv.y += o[1];
      hv.z += o[2];
      hv.w += o[3];
      *(float4*)hp = hv;
      const uint2 g = g_in;
      uint2 pk;
      pk.x = f2bf(hv.x * bf2f(g.x & 0xFFFFu)) | (f2bf(hv.y * bf2f(g.x >> 16)) << 16);
      pk.y = f2bf(hv.z * bf2f(g.y & 0xFFFFu)) | (f2bf(hv.w * bf2f(g.y >> 16)) << 16);
      *(uint2*)(a.a_out + (size_t)m * N + n0) = pk;
      ss = hv.x * hv.x + hv.y * hv.y + hv.z * hv.z + hv.w * hv.w;
    }
    ss += __shfl_xor(ss, 1);
    ss += __shfl_xor(ss, 2);
    if (valid && (c4 & 3) == 0) a.ss_out[(size_t)m * a.ld_ss + n0 / 16] = ss;
  } else {  // kEpiQkv
    if (!valid) return;
    const int D = a.head_dim, qd = a.n_q_heads * D, kd = a.n_kv_heads * D;
    const int sec = n0 < qd ? 0 : n0 < qd + kd ? 1 : 2;
    const int c0 = sec == 0 ? n0 : sec == 1 ? n0 - qd : n0 - qd - kd;
    const int head = c0 / D, d = c0 % D;
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] *= rho;
    if (sec < 2) {
#pragma unroll
      for (int pr = 0; pr < 2; ++pr) {
        const float c = pr ? rope.z : rope.x, s_ = pr ? rope.w : rope.y;
        const float x0 = o[2 * pr], x1 = o[2 * pr + 1];
        o[2 * pr] = x0 * c - x1 * s_;
        o[2 * pr + 1] = x0 * s_ + x1 * c;
      }
    }
    uint32_t b[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) b[q] = f2bf(o[q]);
    if (a.qkv_trace)
      *(uint2*)(a.qkv_trace + (size_t)m * (qd + 2 * kd) + n0) = make_uint2(b[0] | (b[1] << 16), b[2] | (b[3] << 16));
    if (sec == 0) {
      const size_t qo = (((size_t)m * a.n_layers + a.layer) * a.n_q_heads + head) * D + d;
      *(uint2*)(a.q_out + qo) = make_uint2(b[0] | (b[1] << 16), b[2] | (b[3] << 16));
    } else {
      const int slot = pos % kPage;
      const size_t base = (((size_t)a.layer * a.max_pages + phys) * a.n_kv_heads + head) * kPage * D;
      uint16_t* pool = sec == 1 ? a.kpool : a.vpool;
#pragma unroll
      for (int q = 0; q < 4; ++q) pool[base + (sec == 1 ? kswz(slot, d + q) : vswz(slot, d + q))] = (uint16_t)b[q];
    }
  }
}

// Token embedding of every sequence's new token (the query's token), the first
// layer's norm input bf16(h * g) and the per-16-column sums of h^2.
__global__ __launch_bounds__(256) void k_embed(EmbedArgs a) {
  const int s = blockIdx.x;
  const int tok = min(max(a.tokens[(size_t)a.seq_query[s] * a.tok_stride], 0), a.vocab - 1);
  const uint16_t* e = a.embed + (size_t)tok * a.hidden;
  const int n4 = a.hidden / 4;  // a multiple of 64: a wave's groups are all in range or all out
  // the loads of up to U 4-element groups per thread go out before any store
  // (the stores could alias the inputs as far as the compiler knows)
  constexpr int U = 4;
  for (int j0 = threadIdx.x; j0 < n4; j0 += U * 256) {
    uint2 evs[U], gs[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = min(j0 + u * 256, n4 - 1);
      evs[u] = *(const uint2*)(e + 4 * j);
      gs[u] = *(const uint2*)(a.g + 4 * j);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u * 256;
      if (j < n4) {
        const uint2 ev = evs[u], g = gs[u];
        const float h0 = bf2f(ev.x & 0xFFFFu), h1 = bf2f(ev.x >> 16), h2 = bf2f(ev.y & 0xFFFFu),
                    h3 = bf2f(ev.y >> 16);
        *(float4*)(a.h + (size_t)s * a.hidden + 4 * j) = make_float4(h0, h1, h2, h3);
        uint2 pk;
        pk.x = f2bf(h0 * bf2f(g.x & 0xFFFFu)) | (f2bf(h1 * bf2f(g.x >> 16)) << 16);
        pk.y = f2bf(h2 * bf2f(g.y & 0xFFFFu)) | (f2bf(h3 * bf2f(g.y >> 16)) << 16);
        *(uint2*)(a.a_out + (size_t)s * a.hidden + 4 * j) = pk;
        float ss = h0 * h0 + h1 * h1 + h2 * h2 + h3 * h3;
        ss += __shfl_xor(ss, 1);
        ss += __shfl_xor(ss, 2);
        if ((j & 3) == 0) a.ss_out[(size_t)s * a.ld_ss + j / 4] = ss;
      }
    }
  }
}

// Metadata of a prefill chunk's rows (see PrefillMetaArgs): one block per row.
__global__ __launch_bounds__(64) void k_prefill_meta(PrefillMetaArgs a) {
  const int ng = (a.T + a.tq - 1) / a.tq;  // rows (token groups) per sequence
  const int r = blockIdx.x, s = r / ng, j = r - s * ng;
  const int i = min(a.tq * j + a.tq, a.T) - 1;  // the group's last token
  if (threadIdx.x == 0) {
    a.len0_out[r] = a.len0[s] + i;
    if (a.tok_map) a.tok_map[r] = a.seq_query[s] * a.n_tokens + a.i0 + i;
  }
  for (int p = threadIdx.x; p < a.maxpps; p += 64)
    a.page_table_out[(size_t)r * a.maxpps + p] = a.page_table[(size_t)s * a.maxpps + p];
}

// Tokens [start, start + count) of one sequence and layer out of the paged pool
// into contiguous [count][Hkv][D] rows: one block per (token, kv-head), one
// thread per dimension.
__global__ __launch_bounds__(128) void k_read_cache(ReadCacheArgs a) {
  const int i = blockIdx.x, g = blockIdx.y, d = threadIdx.x;
  if (d >= a.head_dim) return;
  const int tok = a.start + i, D = a.head_dim;
  const int phys = a.page_table[(size_t)a.seq * a.maxpps + tok / kPage];
  const int t = tok % kPage;
  const size_t base = (((size_t)a.layer * a.max_pages + phys) * a.n_kv_heads + g) * kPage * D;
  const size_t o = ((size_t)i * a.n_kv_heads + g) * D + d;
  if (a.bf16) {
    ((uint16_t*)a.k_out)[o] = ((const uint16_t*)a.kpool)[base + kswz(t, d)];
    ((uint16_t*)a.v_out)[o] = ((const uint16_t*)a.vpool)[base + vswz(t, d)];
  } else {
    ((float*)a.k_out)[o] = ((const float*)a.kpool)[base + (size_t)t * D + d];
    ((float*)a.v_out)[o] = ((const float*)a.vpool)[base + (size_t)t * D + d];
  }
}

// XOR of every 32-bit word of n16 16-byte units, read with the decode kernels'
// streaming loads: eight loads in flight per lane, grid-stride, one wave-level
// fold and one vector atomic per wave.
__global__ __launch_bounds__(256) void k_stream_read(const uint4* __restrict__ p, size_t n16, uint32_t* out) {
  constexpr int U = 8;
  const size_t stride = (size_t)gridDim.x * 256;
  uint32_t x = 0u;
  size_t i = blockIdx.x * (size_t)256 + threadIdx.x;
  for (; i + (U - 1) * stride < n16; i += U * stride) {
    uint4 v[U];
#pragma unroll
    for (int j = 0; j < U; ++j) v[j] = ld_w<true>(p + i + j * stride);
#pragma unroll
    for (int j = 0; j < U; ++j) x ^= v[j].x ^ v[j].y ^ v[j].z ^ v[j].w;
  }
  for (; i < n16; i += stride) {
    const uint4 v = ld_w<true>(p + i);
    x ^= v.x ^ v.y ^ v.z ^ v.w;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x ^= (uint32_t)__shfl_xor((int)x, o);
  if ((threadIdx.x & 63) == 0) atomicXor(out, x);
}

// RoPE table: (cos, sin) of pos * theta^(-2i/D) in fp64, rounded to fp32.
__global__ __launch_bounds__(256) void k_rope_table(float2* out, int P, int D, double log2_theta) {
  const int half = D / 2;
  for (size_t e = blockIdx.x * (size_t)256 + threadIdx.x; e < (size_t)P * half; e += (size_t)gridDim.x * 256) {
    const int pos = (int)(e / half), i = (int)(e % half);
    const double ang = (double)pos * exp2(-(2.0 * i / D) * log2_theta);
    double sn, cs;
    sincos(ang, &sn, &cs);
    out[e] = make_float2((float)cs, (float)sn);
  }
}

// rho[m] = 1/sqrt(sum_p ss[m][p] * inv_dim + eps) (row stride ld).
__global__ __launch_bounds__(256) void k_rho(const float* ss, int parts, int ld, int M, float inv_dim, float eps,
                                             float* rho) {
  // one wave per row: its partial sums are contiguous
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (m >= M) return;
  float t = 0.f;
  for (int p = lane; p < parts; p += 64) t += ss[(size_t)m * ld + p];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) t += __shfl_xor(t, o);
  if (lane == 0) rho[m] = 1.0f / sqrtf(t * inv_dim + eps);
}

}  // namespace

// ------------------------------------------------------------------ launchers


namespace {
// Launch; timing events, when given, are attached to the dispatch itself
// (start when the kernel begins, stop when it completes), so they measure the
// kernel and not the queue around it.
template <typename Kern, typename... Args>
hipError_t go(Kern kernel, dim3 grid, dim3 block, size_t shm, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1,
              Args... args) {
  if (ev0 || ev1) hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)shm, st, ev0, ev1, 0u, args...);
  else hipLaunchKernelGGL(kernel, grid, block, shm, st, args...);
  return hipGetLastError();
}
hipEvent_t t0(const Timing* tm) { return tm ? tm->start : nullptr; }
hipEvent_t t1(const Timing* tm) { return tm ? tm->stop : nullptr; }
}  // namespace

hipError_t launch_fill_i32(int32_t* p, int32_t v, size_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  const int blocks = (int)((n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024);
  k_fill_i32<<<blocks, 256, 0, st>>>(p, v, n);
  return hipGetLastError();
}

hipError_t launch_zero_bytes(void* p, size_t nbytes, hipStream_t st) {
  const size_t n = nbytes / 4;
  if (n == 0) return hipSuccess;
  const int blocks = (int)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
  k_zero_u32<<<blocks, 256, 0, st>>>((uint32_t*)p, n);
  return hipGetLastError();
}

hipError_t launch_load(const LoadArgs& a, int n_items, bool bf16, hipStream_t st, const Timing* tm) {
  if (n_items == 0) return hipSuccess;
  dim3 grid(n_items, a.n_layers);
  if (bf16) return go(k_load<true>, grid, dim3(256), 0, st, t0(tm), t1(tm), a);
  return go(k_load<false>, grid, dim3(256), 0, st, t0(tm), t1(tm), a);
}

hipError_t launch_append(const AppendArgs& a, bool bf16, hipStream_t st, const Timing* tm) {
  const int blocks = (a.k_new ? a.n_seqs * a.n_layers : 0) + a.n_seqs;  // no K/V rows given: planning only
  if (bf16) return go(k_append<true>, dim3(blocks), dim3(128), 0, st, t0(tm), t1(tm), a);
  return go(k_append<false>, dim3(blocks), dim3(128), 0, st, t0(tm), t1(tm), a);
}

hipError_t launch_attn(const AttnArgs& a, int n_blocks, int head_dim, bool bf16, hipStream_t st, const Timing* tm) {
  if (bf16) {
    const bool s = !a.kv_reread;
    // decode at head dim 128: a 3-page ring (two pages in flight) measured
    // faster than 4 pages (33.7 against 34.2 us at 33 caches x 32 layers): fewer
    // loads past each chunk's end for the same two waves per SIMD
    if (head_dim == 128)
      return s ? go(k_attn_bf16<128, 3, true>, dim3(n_blocks), dim3(64), 0, st, t0(tm), t1(tm), a)
               : go(k_attn_bf16<128, 4, false>, dim3(n_blocks), dim3(64), 0, st, t0(tm), t1(tm), a);
    if (head_dim == 64)
      return s ? go(k_attn_bf16<64, 4, true>, dim3(n_blocks), dim3(64), 0, st, t0(tm), t1(tm), a)
               : go(k_attn_bf16<64, 4, false>, dim3(n_blocks), dim3(64), 0, st, t0(tm), t1(tm), a);
    return hipErrorInvalidValue;
  }
  return go(k_attn_f32, dim3(n_blocks), dim3(64), 0, st, t0(tm), t1(tm), a, head_dim);
}

int attn_blocks_per_cu(int head_dim, bool bf16) {
  int n = 0;
  hipError_t e;
  if (bf16 && head_dim == 128) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_attn_bf16<128, 3, true>, 64, 0);
  else if (bf16) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_attn_bf16<64, 4, true>, 64, 0);
  else e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_attn_f32, 64, 0);
  return (e == hipSuccess && n > 0) ? n : 8;
}

hipError_t launch_attn_combine(const AttnArgs& a, int head_dim, int max_splits, bool bf16, hipStream_t st,
                               const Timing* tm) {
  const int blocks = a.n_seqs * a.n_kv_heads;
  (void)max_splits;
  if (bf16) {
    const int items = blocks * a.group;
    // the prefill's token groups (kv_reread): a wave per (item, kv-head)
    const dim3 mq((blocks + 3) / 4);
    if (head_dim == 128)
      return a.kv_reread ? go(k_attn_combine_mq<128>, mq, dim3(256), 0, st, t0(tm), t1(tm), a)
                         : go(k_attn_combine_bf16<128>, dim3(items), dim3(64), 0, st, t0(tm), t1(tm), a);
    if (head_dim == 64)
      return a.kv_reread ? go(k_attn_combine_mq<64>, mq, dim3(256), 0, st, t0(tm), t1(tm), a)
                         : go(k_attn_combine_bf16<64>, dim3(items), dim3(64), 0, st, t0(tm), t1(tm), a);
    return hipErrorInvalidValue;
  }
  return go(k_attn_combine_f32, dim3(blocks), dim3(128), 0, st, t0(tm), t1(tm), a, head_dim);
}

hipError_t launch_pack_lm_head(const void* w, void* wp, int V, int K, bool bf16, hipStream_t st) {
  if (!bf16) return hipMemcpyAsync(wp, w, (size_t)V * K * 4, hipMemcpyDeviceToDevice, st);
  const size_t nvb = (size_t)(V + 15) / 16, ks = (size_t)K / 64;
  k_pack_w_bf16<<<2048, 256, 0, st>>>((const uint16_t*)w, (uint16_t*)wp, V, K, 1, 0, kLmKMajor ? 1 : ks,
                                      kLmKMajor ? nvb : 1);
  return hipGetLastError();
}

hipError_t launch_pack_tiles(const void* w, void* wp, int rows, int K, int stride, int offset, int n_tiles,
                             hipStream_t st) {
  k_pack_w_bf16<<<2048, 256, 0, st>>>((const uint16_t*)w, (uint16_t*)wp, rows, K, stride, offset,
                                      kProjKMajor ? 1 : (size_t)K / 64, kProjKMajor ? (size_t)n_tiles : 1);
  return hipGetLastError();
}

int proj_tiles_per_wave(int n_tiles) { return n_tiles >= 1024 ? 2 : 1; }

size_t proj_lds_bytes(int rows, int K, int ksplit) {
  const int n = (K / 64 + ksplit - 1) / ksplit;  // longest slice
  return (size_t)rows * (64 * n + 8) * 2;
}

namespace {
// the K-slice sum and epilogue of a projection (ksplit <= kProjMaxSplit)
template <int EPI>
hipError_t launch_reduce_epi(const GemmArgs& a, dim3 g, hipStream_t st, hipEvent_t ev1) {
  const dim3 b(256);
  static_assert(kProjMaxSplit == 16, "slice-count instantiations below");
  if (a.ksplit <= 1) return go(k_proj_reduce<EPI, 1>, g, b, 0, st, nullptr, ev1, a);
  if (a.ksplit <= 2) return go(k_proj_reduce<EPI, 2>, g, b, 0, st, nullptr, ev1, a);
  if (a.ksplit <= 4) return go(k_proj_reduce<EPI, 4>, g, b, 0, st, nullptr, ev1, a);
  if (a.ksplit <= 8) return go(k_proj_reduce<EPI, 8>, g, b, 0, st, nullptr, ev1, a);
  return go(k_proj_reduce<EPI, 16>, g, b, 0, st, nullptr, ev1, a);
}
hipError_t launch_reduce(const GemmArgs& a, GemmEpi epi, hipStream_t st, hipEvent_t ev1) {
  if (a.ksplit < 1 || a.ksplit > kProjMaxSplit) return hipErrorInvalidValue;
  const int outc = epi == kEpiSwiglu ? 8 * a.n_tiles : 16 * a.n_tiles;  // output columns
  const dim3 g((outc / 4 + 255) / 256, a.M);
  switch (epi) {
    case kEpiQkv: return launch_reduce_epi<kEpiQkv>(a, g, st, ev1);
    case kEpiResid: return launch_reduce_epi<kEpiResid>(a, g, st, ev1);
    case kEpiSwiglu: return launch_reduce_epi<kEpiSwiglu>(a, g, st, ev1);
    default: return hipErrorInvalidValue;
  }
}
}  // namespace

hipError_t launch_gemm(const GemmArgs& a, GemmEpi epi, hipStream_t st, const Timing* tm) {
  // up to 48 rows (three 16-row groups in the matrix cores' N dimension); more
  // rows are dense contractions for the library GEMM (launch_proj_epilogue)
  if (a.K % 64 != 0 || a.M < 1 || a.M > kLmRowsPad || a.n_tiles < 1) return hipErrorInvalidValue;
  if (epi == kEpiSwiglu && a.n_tiles % 2) return hipErrorInvalidValue;
  if (a.ksplit < 1 || a.ksplit > a.K / 64) return hipErrorInvalidValue;
  const int NT = a.M <= 16 ? 1 : a.M <= 32 ? 2 : 3;
  const int tpw = proj_tiles_per_wave(a.n_tiles);
  const size_t lds = proj_lds_bytes(a.M, a.K, a.ksplit);
  if (lds > kProjMaxLds) return hipErrorInvalidValue;
  const dim3 b(64 * kProjWaves);
  const dim3 g((a.n_tiles + kProjWaves * tpw - 1) / (kProjWaves * tpw) * a.ksplit);
  hipError_t e;
  if (tpw == 1)
    e = NT == 1 ? go(k_proj<1, 1>, g, b, lds, st, t0(tm), nullptr, a)
        : NT == 2 ? go(k_proj<2, 1>, g, b, lds, st, t0(tm), nullptr, a)
                  : go(k_proj<3, 1>, g, b, lds, st, t0(tm), nullptr, a);
  else
    e = NT == 1 ? go(k_proj<1, 2>, g, b, lds, st, t0(tm), nullptr, a)
        : NT == 2 ? go(k_proj<2, 2>, g, b, lds, st, t0(tm), nullptr, a)
                  : go(k_proj<3, 2>, g, b, lds, st, t0(tm), nullptr, a);
  if (e != hipSuccess) return e;
  return launch_reduce(a, epi, st, t1(tm));
}

hipError_t launch_proj_epilogue(const GemmArgs& a, GemmEpi epi, hipStream_t st, const Timing* tm) {
  if (a.M < 1 || a.n_tiles < 1 || (epi == kEpiSwiglu && a.n_tiles % 2)) return hipErrorInvalidValue;
  GemmArgs r = a;
  r.ksplit = 1;
  if (epi != kEpiResid && a.ss_in && a.rho_rows) {
    const hipError_t e = launch_rho(a.ss_in, a.ss_parts, a.ld_ss, a.M, a.inv_norm_dim, a.eps, a.rho_rows, st);
    if (e != hipSuccess) return e;
    r.rho_in = a.rho_rows;
  }
  return launch_reduce(r, epi, st, t1(tm));
}

hipError_t launch_rope_table(float2* out, int positions, int head_dim, double log2_theta, hipStream_t st) {
  if (positions < 1 || head_dim < 4 || head_dim % 4) return hipErrorInvalidValue;
  const size_t n = (size_t)positions * (head_dim / 2);
  return go(k_rope_table, dim3((unsigned)std::min<size_t>((n + 255) / 256, 2048)), dim3(256), 0, st, nullptr, nullptr,
            out, positions, head_dim, log2_theta);
}

hipError_t launch_embed(const EmbedArgs& a, int n_seqs, hipStream_t st, const Timing* tm) {
  if (a.hidden % 256 != 0) return hipErrorInvalidValue;
  return go(k_embed, dim3(n_seqs), dim3(256), 0, st, t0(tm), t1(tm), a);
}

hipError_t launch_prefill_meta(const PrefillMetaArgs& a, hipStream_t st) {
  if (a.tq < 1) return hipErrorInvalidValue;
  return go(k_prefill_meta, dim3(a.n_seqs * ((a.T + a.tq - 1) / a.tq)), dim3(64), 0, st, nullptr, nullptr, a);
}

hipError_t launch_read_cache(const ReadCacheArgs& a, hipStream_t st) {
  return go(k_read_cache, dim3(a.count, a.n_kv_heads), dim3(128), 0, st, nullptr, nullptr, a);
}

hipError_t launch_rho(const float* ss, int parts, int ld, int M, float inv_dim, float eps, float* rho,
                      hipStream_t st) {
  return go(k_rho, dim3((M + 3) / 4), dim3(256), 0, st, nullptr, nullptr, ss, parts, ld, M, inv_dim, eps,
            rho);
}

int lmhead_wide_tiles(int M, int V, int K) {
  if (M <= kLmRowsPad || M > kLmWideMaxRows || K % 256 != 0) return 0;
  if ((size_t)((V + 15) / 16) * 16 * K * 2 >= 0x7FFFFFFFull) return 0;  // 32-bit buffer offsets into W
  const int mt = (M + 15) / 16;
  return mt <= 8 ? 4 : mt <= 12 ? 6 : 9;  // the instantiated tile counts per row half
}

int lmhead_fused_nblk(int M, int V) {
  if (M <= kLmRowsPad) return (V + 255) / 256;         // 48-row kernel: 256 columns per block
  if (M <= 32 * kLmRowsMTW) return (V + 127) / 128;    // many-row kernel: 128 columns per block
  return 0;
}

hipError_t launch_lmhead(const LmArgs& a0, bool bf16, hipStream_t st, const Timing* tm) {
  LmArgs a = a0;
  if (bf16) {
    const int nvb = (a.V + 15) / 16;
    a.w_vb = kLmKMajor ? 128 : (size_t)(a.K / 64) * 128;
    a.w_ks = kLmKMajor ? (size_t)nvb * 128 : 128;
    const bool fused = a.fuse_part != nullptr;
    if (fused && lmhead_fused_nblk(a.M, a.V) == 0) return hipErrorInvalidValue;
    const int mtk = lmhead_wide_tiles(a.M, a.V, a.K);
    if (mtk > 0 && a.x_packed && a.rho_buf) {
      // many rows: W streamed once for all of them; x packed into operand order
      // (and the row scales) first
      hipError_t e = go(k_pack_x, dim3((32 * mtk + 3) / 4), dim3(256), 0, st, t0(tm), nullptr, (const uint16_t*)a.x,
                        a.M, a.K, 2 * mtk, a.rms, (uint4*)a.x_packed, a.rho_buf);
      if (e != hipSuccess) return e;
      if (!a.rho_in) a.rho_in = a.rho_buf;
      a.x = a.x_packed;
      const dim3 g((nvb + 15) / 16), b(512);
      // up to 128 rows the x stages are small enough for eight of them (and a
      // 16-slot W ring), when the hidden size is a multiple of 8 steps
      const bool deep = mtk == 4 && a.K % 512 == 0;
#define PCED_WIDE(MT, NS)                                                                                    \
  return fused ? go(k_lmhead_wide_bf16<MT, NS, true>, g, b, 0, st, nullptr, t1(tm), a)                       \
               : go(k_lmhead_wide_bf16<MT, NS, false>, g, b, 0, st, nullptr, t1(tm), a);
      if (deep) PCED_WIDE(4, 8)
      if (mtk == 4) PCED_WIDE(4, 4)
      if (mtk == 6) PCED_WIDE(6, 4)
      if (mtk == 9) PCED_WIDE(9, 4)
#undef PCED_WIDE
    }
    if (a.M > kLmRowsPad && a.M <= 32 * kLmRowsMTW) {  // many rows: W streamed once for all of them
      constexpr int VTW = 2, WPB = 8;
      const int blocks = (nvb + WPB / 2 * VTW - 1) / (WPB / 2 * VTW);
      const dim3 g(blocks), b(64 * WPB);
      if (a.K % 128 != 0) return hipErrorInvalidValue;  // bf16 hidden sizes are multiples of 256
      if (fused) return go(k_lmhead_rows_bf16<VTW, kLmRowsMTW, 2, WPB, true>, g, b, 0, st, t0(tm), t1(tm), a);
      return go(k_lmhead_rows_bf16<VTW, kLmRowsMTW, 2, WPB, false>, g, b, 0, st, t0(tm), t1(tm), a);
    }
    // up to 48 rows, or beyond the many-row kernel: 48-row groups, the groups of
    // one vocab chunk together on one XCD so that W comes from HBM once
    constexpr int VT = 4, NT = 3;
    if (fused && a.M > 16 * NT) return hipErrorInvalidValue;  // the fused epilogue covers one row group
    const int chunks = (nvb + 4 * VT - 1) / (4 * VT);
    LmArgs b = a;
    b.row_groups = (a.M + 16 * NT - 1) / (16 * NT);
    const int blocks = b.row_groups > 1 ? (chunks + 7) / 8 * 8 * b.row_groups : chunks;
    // row groups > 1 share each W tile through the XCD's L2: plain loads
    if (b.row_groups > 1)
      return fused ? go(k_lmhead_bf16<VT, NT, true, false>, dim3(blocks), dim3(256), 0, st, t0(tm), t1(tm), b)
                   : go(k_lmhead_bf16<VT, NT, false, false>, dim3(blocks), dim3(256), 0, st, t0(tm), t1(tm), b);
    return fused ? go(k_lmhead_bf16<VT, NT, true, true>, dim3(blocks), dim3(256), 0, st, t0(tm), t1(tm), b)
                 : go(k_lmhead_bf16<VT, NT, false, true>, dim3(blocks), dim3(256), 0, st, t0(tm), t1(tm), b);
  }
  return go(k_lmhead_f32, dim3((a.V + 255) / 256), dim3(256), 0, st, t0(tm), t1(tm), a);
}

hipError_t launch_beta(const BetaArgs& a, int n_seqs, int n_exp, hipStream_t st, const Timing* tm) {
  hipError_t e = go(k_beta_lse, dim3(a.nchunk, n_seqs), dim3(256), 0, st, t0(tm), nullptr, a);
  if (e != hipSuccess) return e;
  e = go(k_beta_jsd, dim3(a.nchunk, n_exp), dim3(256), 0, st, nullptr, nullptr, a);
  if (e != hipSuccess) return e;
  return go(k_beta_final, dim3(n_exp), dim3(64), 0, st, nullptr, t1(tm), a, n_exp);
}

int fuse_slice(int V, int n_queries, int num_cus) {
  // 1024-token slices unless that leaves fewer work-groups than compute units
  return (long)((V + 1023) / 1024) * n_queries >= num_cus ? 1024 : 512;
}

template <int SW>
hipError_t launch_fuse_sw(const FuseArgs& a, dim3 g, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
  const bool vec = a.V % 4 == 0 && a.V >= 4;
  // rows per load batch: a wave's quarter of the experts in one batch up to 16 or 32 experts
  if ((a.max_n + 3) / 4 <= 4)
    return vec ? go(k_fuse<true, 4, SW>, g, dim3(256), 0, st, e0, e1, a)
               : go(k_fuse<false, 4, SW>, g, dim3(256), 0, st, e0, e1, a);
  return vec ? go(k_fuse<true, 8, SW>, g, dim3(256), 0, st, e0, e1, a)
             : go(k_fuse<false, 8, SW>, g, dim3(256), 0, st, e0, e1, a);
}

hipError_t launch_fuse(const FuseArgs& a, int n_queries, hipStream_t st, const Timing* tm, const Timing* tm_merge) {
  // a.nblk: slices of fuse_slice() tokens
  const int sw = (a.V + a.nblk - 1) / a.nblk > 512 ? 1024 : 512;
  const dim3 g(a.nblk, n_queries);
  hipError_t e = sw == 1024 ? launch_fuse_sw<1024>(a, g, st, t0(tm), t1(tm)) : launch_fuse_sw<512>(a, g, st, t0(tm), t1(tm));
  if (e != hipSuccess) return e;
  return go(k_fuse_final, dim3(n_queries), dim3(kFuseBlock), 0, st, t0(tm_merge), t1(tm_merge), a);
}

hipError_t launch_beta_mean(const BetaArgs& a, int n_queries, hipStream_t st) {
  return go(k_beta_mean, dim3(n_queries), dim3(64), 0, st, nullptr, nullptr, a);
}

hipError_t launch_agg(const AggArgs& a, int n_exp, int n_queries, hipStream_t st, const Timing* tm) {
  hipError_t e = go(k_agg_lse, dim3(a.nchunk, n_exp), dim3(256), 0, st, t0(tm), nullptr, a);
  if (e != hipSuccess) return e;
  e = go(k_agg_lse_final, dim3((n_exp + 255) / 256), dim3(256), 0, st, nullptr, nullptr, a, n_exp);
  if (e != hipSuccess) return e;
  return go(k_agg, dim3(a.nblk, n_queries), dim3(kFuseBlock), 0, st, nullptr, t1(tm), a);
}

hipError_t launch_fuse_final(const FuseArgs& a, int n_queries, hipStream_t st, const Timing* tm) {
  return go(k_fuse_final, dim3(n_queries), dim3(kFuseBlock), 0, st, t0(tm), t1(tm), a);
}

hipError_t launch_synth(const SynthArgs& a, int n_seqs, hipStream_t st, const Timing* tm) {
  const int blocks = n_seqs * a.n_layers;
  if (a.bf16) return go(k_synth<true>, dim3(blocks), dim3(256), 0, st, t0(tm), t1(tm), a);
  return go(k_synth<false>, dim3(blocks), dim3(256), 0, st, t0(tm), t1(tm), a);
}

hipError_t launch_stream_read(const void* src, size_t nbytes, uint32_t* xor_out, int num_cus, hipStream_t st) {
  hipError_t e = go(k_zero_u32, dim3(1), dim3(64), 0, st, nullptr, nullptr, xor_out, (size_t)1);
  if (e != hipSuccess || nbytes == 0) return e;
  const size_t n16 = nbytes / 16;
  const size_t want = (n16 + 2047) / 2048;  // eight 16-byte loads per lane
  const unsigned blocks = (unsigned)std::max<size_t>(1, std::min<size_t>(want, (size_t)num_cus * 8));
  return go(k_stream_read, dim3(blocks), dim3(256), 0, st, nullptr, nullptr, (const uint4*)src, n16, xor_out);
}

hipError_t launch_copy_rows(const void* src, void* dst, size_t nbytes, hipStream_t st) {
  return hipMemcpyAsync(dst, src, nbytes, hipMemcpyDeviceToDevice, st);
}

// ------------------------------------------------- allocation-free scratch

// Device scratch of the allocation-free entry point (pced_lmhead_noalloc): a
// library-owned array instead of caller workspace, one copy per GPU the library
// runs on, held until the process ends. In host code its name is only a
// host-side stand-in: kernels and copies get the device address that
// hipGetSymbolAddress returns for the current device (kept per device).
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t noalloc_scratch(void** out) {
  *out = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {  // first use on this device, with the device current
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace pced
