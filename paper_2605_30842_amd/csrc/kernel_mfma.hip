// Matrix-core (MFMA) decode-attention kernel for bf16 caches on gfx950.
//
// One work item = one (split j, KV head hk, sequence b), run by one
// workgroup: in the grid form one workgroup per item, in the work-queue form
// persistent workgroups that take items from a queue. The 4 waves take
// 32-token tiles of the split in turn. Per tile a wave computes
//   S^T[token, head] = K_tile . Q^T    with v_mfma_f32_16x16x32_bf16
// (16 tokens x 16 head columns per instruction; the G real heads of the GQA
// group occupy the first G columns), runs the online softmax on the scores
// in registers, and accumulates
//   O[head, d] += P[head, token] . V_tile[token, d]
// again with 16x16x32 MFMAs. P is split as P = P_hi + P_lo, both bf16, and
// both halves are multiplied (two MFMAs), so the weights keep about 16
// significant bits instead of bf16's 8.
//
// Operand layouts (lane = 16 * g + c, c in 0..15, g in 0..3):
//   MFMA 16x16x32 reads, for A, row c and reduction elements 8g..8g+7 of the
//   lane; for B, column c and the same reduction elements; it returns
//   D[4g + r][c] in accumulator register r.
//   QK:  A = K rows (token c of the sub-tile), reduction = head_dim slice
//        32kb + 8g .. +8 -> one 16-byte load per (sub-tile, kb).
//        B = Q rows (head c), same slice. Result: lane holds the score of
//        head c for tokens 4g + r of each 16-token sub-tile.
//   PV:  A = P: lane already holds head c's weights for the 8 tokens
//        {16s + 4g + r}; they become reduction elements e = 4s + r.
//        B = V: the same 8 tokens, column c standing for d = NT*c + n in
//        n-tile n (NT = D/16). Loading V row (16s + 4g + r), bytes
//        [2*NT*c, 2*NT*(c+1)) gives every n-tile's element at once, and
//        those loads read whole 256-byte rows with 16 consecutive lanes.
//        A v_perm per element pair regroups them into MFMA operands.
// The reduction index of an MFMA is a dummy index, so any consistent
// assignment of (lane, element) to tokens or head_dim positions is valid as
// long as A and B use the same one, which they do by construction above.
//
// FP8 caches (OCP E4M3 codes with a per-tensor scale) use the same tiles at
// one byte per element and widen the codes to bf16 in registers before the
// matrix-core steps (exact: every E4M3 value is a bf16 value). The scales
// are folded into the score scale (K) and the final output (V). For the QK
// step a lane's K slice is then its D / 4 consecutive codes (head_dim
// (D / 4) g onward, 16 per 16-byte load): k-block kb is head_dim
// (D / 4) g + 8 kb .. + 8, and the Q operand follows the same assignment.
#include "attn_common.h"

namespace comem {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <int D>
struct VRow;  // per-lane slice of one V row: NT bf16 values
// V rows are read whole by consecutive lanes and never again: load them with
// the non-temporal (streaming) cache policy. K rows are read in two halves
// of a 128-byte line by consecutive instructions, so they keep the default
// policy and the second half hits the line the first half brought in.
constexpr int kStreaming = 2;

template <>
struct VRow<128> {
  u32x4 w;
  __device__ uint32_t word(int i) const { return w[i]; }
  __device__ void load(__amdgpu_buffer_rsrc_t r, uint32_t voff, int soff) {
    w = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kStreaming));
  }
};
template <>
struct VRow<64> {
  u32x2 w;
  __device__ uint32_t word(int i) const { return w[i]; }
  __device__ void load(__amdgpu_buffer_rsrc_t r, uint32_t voff, int soff) {
    w = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, kStreaming));
  }
};

template <int D>
struct Tile {
  static constexpr int KB = D / 32;
  u32x4 k[2][KB];   // [sub-tile][k-block]
  VRow<D> v[2][4];  // [sub-tile][r]
};

__device__ inline bf16x8 as_bf16x8(u32x4 x) { return __builtin_bit_cast(bf16x8, x); }

// The V slice of a row in an FP8 cache: NT one-byte codes.
template <int D>
struct VRow8;
template <>
struct VRow8<128> {
  u32x2 w;
  __device__ void load(__amdgpu_buffer_rsrc_t r, uint32_t voff, int soff) {
    w = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, kStreaming));
  }
};
template <>
struct VRow8<64> {
  uint32_t w;
  __device__ void load(__amdgpu_buffer_rsrc_t r, uint32_t voff, int soff) {
    w = __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, kStreaming);
  }
};

template <int D>
struct Tile8 {
  u32x4 k[2][D / 64];  // [sub-tile][16 codes]: the lane's D / 4 codes of its K row
  VRow8<D> v[2][4];
};

template <int D, bool FP8>
struct TileOf {
  using type = Tile<D>;
};
template <int D>
struct TileOf<D, true> {
  using type = Tile8<D>;
};

// Two E4M3 codes (bytes 0-1, or 2-3 with HIGH) of w as a bf16 pair, low element first.
template <bool HIGH>
__device__ inline uint32_t e4m3_pair_to_bf16(uint32_t w) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, HIGH));
}

// Widen an FP8 tile to the bf16 tile the matrix-core steps read.
template <int D>
__device__ inline void widen_tile(const Tile8<D>& R, Tile<D>& T) {
  constexpr int KB = D / 32;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const uint32_t w0 = R.k[s][kb >> 1][2 * (kb & 1)], w1 = R.k[s][kb >> 1][2 * (kb & 1) + 1];
      T.k[s][kb] = u32x4{e4m3_pair_to_bf16<false>(w0), e4m3_pair_to_bf16<true>(w0), e4m3_pair_to_bf16<false>(w1),
                         e4m3_pair_to_bf16<true>(w1)};
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      if constexpr (D == 128) {
        const u32x2 w = R.v[s][r].w;
        T.v[s][r].w = u32x4{e4m3_pair_to_bf16<false>(w[0]), e4m3_pair_to_bf16<true>(w[0]),
                            e4m3_pair_to_bf16<false>(w[1]), e4m3_pair_to_bf16<true>(w[1])};
      } else {
        T.v[s][r].w = u32x2{e4m3_pair_to_bf16<false>(R.v[s][r].w), e4m3_pair_to_bf16<true>(R.v[s][r].w)};
      }
    }
  }
}

// Page lookups of one split go through LDS: the workgroup copies the split's
// block-table entries there once, so the token loop never waits on them.
constexpr int kMaxSplitPages = 2048;
// Largest batch the work-queue kernel takes (its per-sequence split offsets live in LDS).
constexpr int kMaxQueueBatch = 4096;

enum class Layout { kContig, kPaged, kPagedFine };

template <int D, Layout LAYOUT, bool FP8>
struct Loader {
  using TileT = typename TileOf<D, FP8>::type;
  static constexpr int kElemBytes = FP8 ? 1 : 2;
  const char* kbase;  // K of this (b, hk): contiguous layout already offset to the sequence start
  const char* vbase;
  const int32_t* sm_pages;  // LDS copy of the split's block-table entries (paged layouts)
  int page_first;           // token index of the first entry in sm_pages
  int64_t stride_token;
  int64_t stride_page;
  int page_shift, page_mask;
  int t_end;
  int c, g;
  uint32_t koff;  // c * stride_token + 16 g (FP8: + (D / 4) g)
  uint32_t voff;  // 4 g * stride_token + (NT * c elements)

  // Byte offset of token t from the base; uniform across the wave when t is.
  __device__ int64_t token_offset(int t) const {
    if constexpr (LAYOUT == Layout::kContig) {
      return static_cast<int64_t>(t) * stride_token;
    } else {
      const int page = max(0, sm_pages[(t - page_first) >> page_shift]);  // -1 (outside the pool) reads page 0
      return static_cast<int64_t>(page) * stride_page + static_cast<int64_t>(t & page_mask) * stride_token;
    }
  }

  // A full 32-token tile whose 16-token halves each lie in one page (or the
  // contiguous layout): per half, one buffer descriptor on the half's first
  // row (uniform, in SGPRs) and fixed 32-bit lane offsets. The descriptor's
  // size covers exactly the 16 rows, so the hardware returns zeros instead of
  // touching memory should an offset ever fall outside them. With `repeat`
  // the call only keeps the load count of the pipeline steady: it re-reads
  // the tile's K rows (still cached) into both halves and its data is unused.
  __device__ void load_full(TileT& T, int t0, bool repeat) const {
    constexpr int KB = D / 32;
    const int extent = static_cast<int>(15 * stride_token + kElemBytes * D);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int64_t base = uniform_i64(token_offset(t0 + 16 * s));
      const __amdgpu_buffer_rsrc_t rk =
          __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(kbase + base), 0, extent, kBufferConfig);
      const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<char*>((repeat ? kbase : vbase) + base), 0, extent, kBufferConfig);
      if constexpr (FP8) {
#pragma unroll
        for (int i = 0; i < D / 64; ++i)
          T.k[s][i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rk, koff + 16 * i, 0, 0));
      } else {
#pragma unroll
        for (int kk = 0; kk < KB; ++kk)
          T.k[s][kk] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rk, koff + 64 * kk, 0, 0));
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) T.v[s][r].load(rv, voff, static_cast<int>(r * stride_token));
    }
  }

  // Any tile: per-lane rows; tokens past the end are clamped to the last
  // valid row (their weight is zero), so no byte outside a context is read.
  __device__ void load_any(TileT& T, int t0) const {
    constexpr int KB = D / 32;
    constexpr int VBYTES = kElemBytes * D / 16;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const char* kr = kbase + token_offset(min(t0 + 16 * s + c, t_end - 1)) + (FP8 ? (D / 4) * g : 16 * g);
      if constexpr (FP8) {
#pragma unroll
        for (int i = 0; i < D / 64; ++i) T.k[s][i] = *reinterpret_cast<const u32x4*>(kr + 16 * i);
      } else {
#pragma unroll
        for (int kk = 0; kk < KB; ++kk) T.k[s][kk] = *reinterpret_cast<const u32x4*>(kr + 64 * kk);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const char* vr = vbase + token_offset(min(t0 + 16 * s + 4 * g + r, t_end - 1)) + VBYTES * c;
        T.v[s][r].w = *reinterpret_cast<const decltype(T.v[s][r].w)*>(vr);
      }
    }
  }
};

template <int D>
__device__ inline void compute_tile(const Tile<D>& T, int t0, int t_end, int g,
                                    const bf16x8 (&qop)[D / 32], float scale_log2, float& m_run,
                                    float& l_run, f32x4 (&acc)[D / 16]) {
  constexpr int KB = D / 32;
  constexpr int NT = D / 16;
  // Scores S^T: lane holds head c, tokens t0 + 16s + 4g + r.
  f32x4 sc[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    sc[s] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KB; ++kk)
      sc[s] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(T.k[s][kk]), qop[kk], sc[s], 0, 0, 0);
  }
  float x[8];
  float mt = -INFINITY;
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = t0 + 16 * s + 4 * g + r;
      const float v = t < t_end ? sc[s][r] * scale_log2 : -INFINITY;
      x[4 * s + r] = v;
      mt = fmaxf(mt, v);
    }
  mt = fmaxf(mt, __shfl_xor(mt, 16));
  mt = fmaxf(mt, __shfl_xor(mt, 32));
  // Every tile holds at least one valid token, so m_new is finite.
  const float m_new = fmaxf(m_run, mt);
  const float alpha = fast_exp2(m_run - m_new);
  {
    float ar[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) ar[r] = __shfl(alpha, 4 * g + r);
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[n][r] *= ar[r];
  }
  m_run = m_new;
  float psum = 0.f;
  uint32_t ph[4], pl[4];
#pragma unroll
  for (int e = 0; e < 8; e += 2) {
    const float p0 = fast_exp2(x[e] - m_new);
    const float p1 = fast_exp2(x[e + 1] - m_new);
    psum += p0 + p1;
    const uint32_t b0 = __float_as_uint(p0), b1 = __float_as_uint(p1);
    ph[e / 2] = __builtin_amdgcn_perm(b1, b0, 0x07060302u);  // upper halves: truncated bf16
    // remainders p - hi are exact in fp32; round them to nearest-even bf16
    uint32_t r0 = __float_as_uint(p0 - __uint_as_float(b0 & 0xffff0000u));
    uint32_t r1 = __float_as_uint(p1 - __uint_as_float(b1 & 0xffff0000u));
    r0 += 0x7fffu + ((r0 >> 16) & 1u);
    r1 += 0x7fffu + ((r1 >> 16) & 1u);
    pl[e / 2] = __builtin_amdgcn_perm(r1, r0, 0x07060302u);
  }
  l_run = l_run * alpha + psum;
  const bf16x8 pa_hi = as_bf16x8(u32x4{ph[0], ph[1], ph[2], ph[3]});
  const bf16x8 pa_lo = as_bf16x8(u32x4{pl[0], pl[1], pl[2], pl[3]});
#pragma unroll
  for (int n = 0; n < NT; ++n) {
    const uint32_t sel = (n & 1) ? 0x07060302u : 0x05040100u;
    const int wi = n >> 1;
    u32x4 vb;
    vb[0] = __builtin_amdgcn_perm(T.v[0][1].word(wi), T.v[0][0].word(wi), sel);
    vb[1] = __builtin_amdgcn_perm(T.v[0][3].word(wi), T.v[0][2].word(wi), sel);
    vb[2] = __builtin_amdgcn_perm(T.v[1][1].word(wi), T.v[1][0].word(wi), sel);
    vb[3] = __builtin_amdgcn_perm(T.v[1][3].word(wi), T.v[1][2].word(wi), sel);
    acc[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa_hi, as_bf16x8(vb), acc[n], 0, 0, 0);
    acc[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa_lo, as_bf16x8(vb), acc[n], 0, 0, 0);
  }
}

// compute_tile on a tile as loaded (FP8 tiles are widened first).
template <int D, bool FP8>
__device__ inline void compute_loaded(const typename TileOf<D, FP8>::type& T, int t0, int t_end, int g,
                                      const bf16x8 (&qop)[D / 32], float scale_log2, float& m_run, float& l_run,
                                      f32x4 (&acc)[D / 16]) {
  if constexpr (FP8) {
    Tile<D> W;
    widen_tile<D>(T, W);
    compute_tile<D>(W, t0, t_end, g, qop, scale_log2, m_run, l_run, acc);
  } else {
    compute_tile<D>(T, t0, t_end, g, qop, scale_log2, m_run, l_run, acc);
  }
}

// ctx_lens[b] and, for the contiguous layout, seq_start[b]: both loads are
// issued before either value is used (the empty asm consumes both at once),
// so they share one memory round trip.
template <Layout LAYOUT>
__device__ inline void load_sequence(const AttnParams& p, int b, int& L, int64_t& seq_row) {
  b = uniform_i32(b);  // uniform in every caller
  L = uniform_i32(p.ctx_lens[b]);
  seq_row = LAYOUT == Layout::kContig ? uniform_i64(p.seq_start[b]) : 0;
  asm volatile("" : "+s"(L), "+s"(seq_row));
  L = checked_len(L, p.max_ctx, p.errors);
}

// Shared memory of one workgroup; the page table and the wave states are
// rewritten for every split the workgroup processes.
template <int D, Layout LAYOUT>
struct SplitSmem {
  WaveState<D> ws;
  int32_t pages[LAYOUT == Layout::kContig ? 1 : kMaxSplitPages];
};

// The splits of a sequence of L tokens in the work-queue form. There are
// ceil(L / chunk) of them (one, empty, when L = 0), normally split j = tokens
// [j * chunk, min((j + 1) * chunk, L)), as in the grid form. With short last
// splits (tail_chunk > 0), the last `small` splits, at most a quarter of
// them, cover tail_chunk tokens each (the very last one up to L) and start
// at a multiple of 32; the others share the tokens before them evenly in
// whole 32-token tiles (the first `rem` of them one tile more), so no split
// exceeds 1.25 chunk. The queue hands out every sequence's large splits
// before any short one, so the items taken last are short and workgroups
// finish close together. The ranges depend on L and the plan only, never on
// which workgroup runs them or when.
struct SplitGeometry {
  int nsplit;       // splits of the sequence
  int small;        // short last splits among them
  int small_start;  // first token of the short splits (L without them)
  int q, rem;       // large split j has q tiles, one more if j < rem

  __device__ SplitGeometry(int L, const AttnParams& p) {
    nsplit = L > 0 ? 1 + (L - 1) / p.chunk : 1;
    small = p.tail_chunk > 0 ? min(p.tail_splits, nsplit / 4) : 0;
    small_start = small > 0 ? (L - small * p.tail_chunk) & ~31 : L;
    const int tiles = small_start >> 5;
    q = small > 0 ? tiles / (nsplit - small) : 0;
    rem = small > 0 ? tiles - q * (nsplit - small) : 0;
  }
  __device__ int big() const { return nsplit - small; }

  // Tokens [t0, t1) of split j < nsplit.
  __device__ void range(int j, int L, const AttnParams& p, int& t0, int& t1) const {
    if (small == 0) {
      t0 = j * p.chunk;
      t1 = t0 + min(L - t0, p.chunk);
    } else if (j < big()) {
      t0 = 32 * (j * q + min(j, rem));
      t1 = t0 + 32 * (q + (j < rem ? 1 : 0));
    } else {
      const int s = j - big();
      t0 = small_start + s * p.tail_chunk;
      t1 = s == small - 1 ? L : t0 + p.tail_chunk;
    }
  }
};

// Attention of the G query heads of KV head hk of sequence b over split j of
// nsplit_b (tokens [t_begin, t_end)), ending with this split's share of the
// log-sum-exp merge. Called by every thread of the workgroup. seq_row is
// seq_start[b] for the contiguous layout (unused when paged); the callers
// load it together with ctx_lens[b], so the two loads cost one round trip
// before the first tile is requested.
//
// With next_item set (work-queue form), thread 0 takes the workgroup's next
// item from the queue once the token loop is done: issued earlier, the queue
// atomic would sit ahead of the tile loads in the in-order memory counter.
template <int D, Layout LAYOUT, bool FP8>
__device__ void attend_split(const AttnParams& p, SplitSmem<D, LAYOUT>& sm, int b, int hk, int j, int nsplit_b,
                             int t_begin, int t_end, int L, int64_t seq_row, int* next_item) {
  using TileT = typename TileOf<D, FP8>::type;
  constexpr int KB = D / 32;
  constexpr int NT = D / 16;
  const int lane = threadIdx.x & 63;
  const int w = uniform_i32(threadIdx.x >> 6);
  const int c = lane & 15, g = lane >> 4;
  const int G = p.group;

  Loader<D, LAYOUT, FP8> ld;
  ld.kbase = p.k + hk * p.stride_head;
  ld.vbase = p.v + hk * p.stride_head;
  if constexpr (LAYOUT == Layout::kContig) {
    const int64_t seq0 = seq_row * p.stride_token;
    ld.kbase += seq0;
    ld.vbase += seq0;
  } else {
    // Entries for tokens [t_begin, t_end); never past ceil(L / page_size).
    ld.page_first = t_begin & ~p.page_mask;
    const int first = t_begin >> p.page_shift;
    const int count = ((t_end - 1) >> p.page_shift) - first + 1;
    const int32_t* row = p.block_table + static_cast<int64_t>(b) * p.max_pages + first;
    for (int i = threadIdx.x; i < count; i += kThreads) sm.pages[i] = checked_page(row[i], p.num_pages, p.errors);
    __syncthreads();
  }
  ld.sm_pages = sm.pages;
  ld.stride_token = p.stride_token;
  ld.stride_page = p.stride_page;
  ld.page_shift = p.page_shift;
  ld.page_mask = p.page_mask;
  ld.t_end = t_end;
  ld.c = c;
  ld.g = g;
  ld.koff = static_cast<uint32_t>(c * p.stride_token + (FP8 ? (D / 4) * g : 16 * g));
  ld.voff = static_cast<uint32_t>(4 * g * p.stride_token + (FP8 ? NT : 2 * NT) * c);

  // Q operand: head c of the group (zero columns past G), slice 32kb + 8g
  // (FP8 caches: (D / 4) g + 8 kb, the slice the lane's K codes cover).
  bf16x8 qop[KB];
  {
    const char* qrow = p.q + (static_cast<int64_t>(b) * p.num_q_heads + hk * G + c) * D * 2;
#pragma unroll
    for (int kk = 0; kk < KB; ++kk) {
      u32x4 qv = u32x4{0u, 0u, 0u, 0u};
      if (c < G) qv = *reinterpret_cast<const u32x4*>(qrow + (FP8 ? (D / 2) * g + 16 * kk : 64 * kk + 16 * g));
      qop[kk] = as_bf16x8(qv);
    }
  }

  float m_run = -INFINITY, l_run = 0.f;
  f32x4 acc[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int ntok = t_end - t_begin;
  const int nfull = ntok >> 5;              // full 32-token tiles
  const int ntiles = (ntok + 31) >> 5;      // including a partial last tile
  // Fused append: the wave that owns the tile of token L - 1 stores its rows
  // first (not when the length was clamped: that row is not the new token's).
  if (p.new_k != nullptr && t_end == L && L > 0 && w == (ntiles - 1) % kWaves && p.ctx_lens[b] == L) {
    int64_t row;
    if constexpr (LAYOUT == Layout::kContig) {
      row = (seq_row + static_cast<int64_t>(L - 1)) * p.stride_token;
    } else {
      row = checked_page_row(p, sm.pages[((L - 1) - ld.page_first) >> p.page_shift], L - 1);
    }
    store_new_token(p, b, hk, row, FP8 ? D / 16 : D / 8, lane);
  }
  int ti = w;
  if constexpr (LAYOUT != Layout::kPagedFine) {
    // Full tiles w, w + 4, ...: while one tile is computed the next is in
    // flight. The prefetch is issued unconditionally (past the last full tile
    // it re-reads cached K rows of the current one) and pinned ahead of the
    // compute, so the compiler waits for exactly the older tile's loads.
    if (ti < nfull) {
      TileT A, B;
      ld.load_full(A, t_begin + 32 * ti, false);
      for (;;) {
        int nx = ti + kWaves;
        ld.load_full(B, t_begin + 32 * (nx < nfull ? nx : ti), nx >= nfull);
        __builtin_amdgcn_sched_barrier(0);
        compute_loaded<D, FP8>(A, t_begin + 32 * ti, t_end, g, qop, p.scale_log2, m_run, l_run, acc);
        if (nx >= nfull) break;
        ti = nx;
        nx = ti + kWaves;
        ld.load_full(A, t_begin + 32 * (nx < nfull ? nx : ti), nx >= nfull);
        __builtin_amdgcn_sched_barrier(0);
        compute_loaded<D, FP8>(B, t_begin + 32 * ti, t_end, g, qop, p.scale_log2, m_run, l_run, acc);
        if (nx >= nfull) break;
        ti = nx;
      }
    }
    ti = nfull;  // the partial tile, if any, belongs to wave nfull % kWaves
    if (ti < ntiles && (ti % kWaves) == w) {
      TileT A;
      ld.load_any(A, t_begin + 32 * ti);
      compute_loaded<D, FP8>(A, t_begin + 32 * ti, t_end, g, qop, p.scale_log2, m_run, l_run, acc);
    }
  } else {
    for (; ti < ntiles; ti += kWaves) {
      TileT A;
      ld.load_any(A, t_begin + 32 * ti);
      compute_loaded<D, FP8>(A, t_begin + 32 * ti, t_end, g, qop, p.scale_log2, m_run, l_run, acc);
    }
  }

  if (next_item != nullptr && threadIdx.x == 0)
    *next_item = static_cast<int>(gridDim.x + atomicAdd(p.tickets + p.queue_slot, 1u));

  // Wave totals: l over the four lane groups; state to LDS.
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  if (g == 0 && c < G) {
    sm.ws.m[w][c] = m_run;
    sm.ws.l[w][c] = l_run;
  }
  // A lane's values of one head are NT consecutive head_dim positions, so
  // they go out as 16-byte stores.
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int h = 4 * g + r;
    if (h < G) {
#pragma unroll
      for (int n = 0; n < NT; n += 4)
        *reinterpret_cast<float4*>(&sm.ws.o[w][h][NT * c + n]) =
            make_float4(acc[n][r], acc[n + 1][r], acc[n + 2][r], acc[n + 3][r]);
    }
  }
  __syncthreads();
  finalize_split<D>(p, sm.ws, b, hk, j, nsplit_b);
}

// One workgroup per (split, KV head, sequence); splits past a sequence's end
// exit. Within a sequence the KV head varies fastest with the linear
// workgroup id, the order in which workgroups are dealt to the XCDs (round
// robin): with 8 KV heads all splits of a head run on one XCD, and the heads
// of a token range are read side by side. The batch-1 32K step with K and V
// in two allocations took 29.1 instead of 30.3 us (27.8 and 27.9 us with the
// recommended placement). Grids of more than 2^24 workgroups per sequence
// keep the direct order (the 32-bit index arithmetic stays exact).
template <int D, Layout LAYOUT, bool FP8>
__global__ __launch_bounds__(kThreads, 2) void decode_mfma_kernel(const AttnParams p) {
  int j = blockIdx.x, hk = blockIdx.y;
  const int b = blockIdx.z;
  if (static_cast<uint64_t>(gridDim.x) * gridDim.y <= (1u << 24)) {
    const uint32_t lin = blockIdx.x + gridDim.x * blockIdx.y;
    hk = static_cast<int>(lin % gridDim.y);
    j = static_cast<int>(lin / gridDim.y);
  }
  int L;
  int64_t seq_row;
  load_sequence<LAYOUT>(p, b, L, seq_row);
  const int nsplit_b = L > 0 ? 1 + (L - 1) / p.chunk : 1;  // even splits (no short last ones)
  if (j >= nsplit_b) return;
  const int t0 = j * p.chunk;
  __shared__ SplitSmem<D, LAYOUT> sm;
  attend_split<D, LAYOUT, FP8>(p, sm, b, hk, j, nsplit_b, t0, t0 + min(L - t0, p.chunk), L, seq_row, nullptr);
}

// In-place prefix sum by one wave: a[i + 1] (counts of sequences 0..n-1)
// becomes the total of the first i + 1 counts, and a[0] = 0.
__device__ inline void wave_prefix_sum(int* a, int n, int lane) {
  int carry = 0;
  for (int base = 0; base < n; base += 64) {
    const int i = base + lane;
    int v = i < n ? a[i + 1] : 0;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int u = __shfl_up(v, o);
      if (lane >= o) v += u;
    }
    if (i < n) a[i + 1] = carry + v;
    carry += __shfl(v, 63);
  }
  if (lane == 0) a[0] = 0;
}

// Sequence b with first[b] <= index < first[b + 1] (first is a prefix sum).
__device__ inline int find_sequence(const int* first, int n, int index) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (first[mid] <= index) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Persistent workgroups that take work items from a queue. The items are
// the large splits of every sequence, in the order (b, j, hk) so that the
// heads of one token range are adjacent and sequences follow each other,
// then the short last splits (SplitGeometry) in the same order. Which
// workgroup runs an item depends on timing, but every item computes the same
// values and the merge order is fixed, so results do not. The queue counter
// and the count of finished workgroups live next to the tickets and return
// to zero when the last workgroup leaves. Faster XCDs and compute units
// simply take more items, and ragged batches need no empty workgroups.
template <int D, Layout LAYOUT, bool FP8>
__global__ __launch_bounds__(kThreads, 2) void decode_mfma_queue_kernel(const AttnParams p, int batch) {
  __shared__ SplitSmem<D, LAYOUT> sm;
  __shared__ int sm_first[kMaxQueueBatch + 1];  // prefix sums of large splits per sequence
  __shared__ int sm_short[kMaxQueueBatch + 1];  // prefix sums of short splits per sequence
  __shared__ int sm_next;
  const int tid = threadIdx.x;
  uint32_t* queue = p.tickets + p.queue_slot;
  uint32_t* finished = queue + 1;

  // Split counts per sequence, then prefix sums (one wave each).
  for (int b = tid; b < batch; b += kThreads) {
    const SplitGeometry geo(checked_len(p.ctx_lens[b], p.max_ctx, nullptr), p);  // reported by load_sequence
    sm_first[b + 1] = geo.big();
    sm_short[b + 1] = geo.small;
  }
  __syncthreads();
  if (tid < 64) wave_prefix_sum(sm_first, batch, tid);
  else if (tid < 128) wave_prefix_sum(sm_short, batch, tid - 64);
  __syncthreads();
  const int total_big = sm_first[batch] * p.num_kv_heads;
  const int total = total_big + sm_short[batch] * p.num_kv_heads;
  // Item blockIdx.x first; later items come from the queue, which hands out
  // gridDim.x, gridDim.x + 1, ... Without more items than workgroups the
  // queue is never touched.
  const bool queued = total > static_cast<int>(gridDim.x);

  int item = blockIdx.x;
  while (item < total) {
    const bool is_big = item < total_big;
    const int index = (is_big ? item : item - total_big) / p.num_kv_heads;
    const int hk = (is_big ? item : item - total_big) - index * p.num_kv_heads;
    const int b = find_sequence(is_big ? sm_first : sm_short, batch, index);
    const int big_b = sm_first[b + 1] - sm_first[b];
    const int j = is_big ? index - sm_first[b] : big_b + index - sm_short[b];
    int L;
    int64_t seq_row;
    load_sequence<LAYOUT>(p, b, L, seq_row);
    const SplitGeometry geo(L, p);
    int t0, t1;
    geo.range(j, L, p, t0, t1);
    attend_split<D, LAYOUT, FP8>(p, sm, b, hk, j, geo.nsplit, t0, t1, L, seq_row, queued ? &sm_next : nullptr);
    __syncthreads();
    item = queued ? sm_next : total;
    __syncthreads();
  }
  if (queued && tid == 0 && atomicAdd(finished, 1u) == gridDim.x - 1) {
    atomicExch(queue, 0u);
    atomicExch(finished, 0u);
  }
}

}  // namespace

using KernelFn = void (*)(AttnParams);
using QueueKernelFn = void (*)(AttnParams, int);

template <int D, bool FP8>
KernelFn pick_layout(bool paged, int page_size) {
  if (!paged) return decode_mfma_kernel<D, Layout::kContig, FP8>;
  return page_size >= 16 ? decode_mfma_kernel<D, Layout::kPaged, FP8> : decode_mfma_kernel<D, Layout::kPagedFine, FP8>;
}

template <int D, bool FP8>
QueueKernelFn pick_queue_layout(bool paged, int page_size) {
  if (!paged) return decode_mfma_queue_kernel<D, Layout::kContig, FP8>;
  return page_size >= 16 ? decode_mfma_queue_kernel<D, Layout::kPaged, FP8>
                         : decode_mfma_queue_kernel<D, Layout::kPagedFine, FP8>;
}

KernelFn select_mfma_kernel(int head_dim, bool paged, int page_size, bool fp8) {
  if (head_dim == 128) return fp8 ? pick_layout<128, true>(paged, page_size) : pick_layout<128, false>(paged, page_size);
  if (head_dim == 64) return fp8 ? pick_layout<64, true>(paged, page_size) : pick_layout<64, false>(paged, page_size);
  return nullptr;
}

QueueKernelFn select_mfma_queue_kernel(int head_dim, bool paged, int page_size, bool fp8) {
  if (head_dim == 128)
    return fp8 ? pick_queue_layout<128, true>(paged, page_size) : pick_queue_layout<128, false>(paged, page_size);
  if (head_dim == 64)
    return fp8 ? pick_queue_layout<64, true>(paged, page_size) : pick_queue_layout<64, false>(paged, page_size);
  return nullptr;
}

int mfma_max_queue_batch() { return kMaxQueueBatch; }

int mfma_max_split_pages() { return kMaxSplitPages; }

}  // namespace comem
