// Matrix-core prefill attention over a cached prefix, bf16 caches, gfx950.
//
// The operation (paper Algorithm 1 and the k-step-off pipeline of Sec. 3.2):
// sequence b holds L_b cached tokens whose last M_b are new (their keys and
// values already appended, as for decode in Sec. 2.2); new token i, at cache
// position L_b - M_b + i, attends over cache tokens 0 .. L_b - M_b + i. A
// cached prefill has a long prefix and few new tokens; an uncached prefill
// (after a summary update) has M_b = L_b, i.e. plain causal attention.
//
// One workgroup takes 128 (new token, query head) rows of one KV head of one
// sequence: 128 / G consecutive new tokens times the G query heads that share
// the KV head, so every K/V tile staged in LDS serves all of them. It has 8
// waves in two halves over the two halves of the key tiles (merged at the
// end); wave w of a half owns rows 32w .. 32w + 31 and, per 64-key tile,
// computes
//   S^T[key, row] = K_tile . Q^T          (v_mfma_f32_32x32x16_bf16)
//   O^T[d, row]  += V_tile^T . P^T        (same instruction)
// with an online softmax in between. In the transposed form a lane owns one
// row in every accumulator: lane = row + 32 * half, where the two halves hold
// different keys (S^T) or different head_dim entries (O^T) of the same row.
// So the causal limit, the running maximum and the rescaling are per lane,
// and the two halves meet in a single xor-32 shuffle per tile.
//
// Operand layouts of v_mfma_f32_32x32x16_bf16 (checked on the device):
//   A[i][k] in lane i + 32 (k / 8), element k % 8;
//   B[k][j] in lane j + 32 (k / 8), element k % 8;
//   D[i][j] in lane j + 32 ((i / 4) % 2), register (i % 4) + 4 (i / 8).
// QK: A = K rows (key i, head_dim slice 16 ks + 8 half .. + 8), B = Q rows
//     (row j, same slice, registers for the whole kernel). Register r of a
//     lane of half h then holds key 8 (r / 4) + 4 h + r % 4 of the block.
// PV: B = P^T takes the probabilities straight from those registers: element
//     e of k-step (block sb, step s2) is register 8 s2 + e, i.e. key
//     32 sb + 16 s2 + 8 (e / 4) + 4 h + e % 4. The reduction index of an MFMA
//     is a dummy index, so A = V^T uses the same key for the same (half,
//     element); row i of n-tile n is head_dim 32 n + i. That operand holds 8
//     keys at one head_dim entry per lane, a transpose of how V is stored; the
//     LDS transpose read (ds_read_b64_tr_b16) produces it directly: within a
//     group of 16 lanes, lane 4a + c receives element c of the 4-element
//     vectors addressed by lanes a, a + 4, a + 8, a + 12 (checked on the
//     device). So lane k of a group addresses key (k / 4) of the step at
//     head_dim 4 (k % 4) onward, and two reads give the 8 keys.
// P is split as P = P_hi + P_lo, both bf16 (the high half truncated, the
// exact remainder rounded to nearest even), and both halves are multiplied,
// so each weight keeps about 16 significant bits: an output is off by at
// most about 2^-15 sum_t w_t |v_t| plus fp32 rounding.
//
// The running maximum moves lazily: it is raised only when a row's new
// maximum exceeds it by more than 2^8 in probability, so the accumulators are
// rescaled rarely and every probability stays below 2^8. A tile's
// probabilities are first taken against the running maximum as it is; the
// tile's own maximum is computed only when a lane's sum of them passes 2^8.
//
// K and V tiles go from global memory straight into LDS (buffer loads with an
// LDS destination), K two tiles and V one tile ahead of the compute, into two
// K and two V slots per half. The descriptors' base and size are uniform per
// 16-row group (one page when pages hold 16 rows or more), so addresses are
// scalar arithmetic and rows past the keys a block needs arrive as zeros. In
// LDS, 16-byte chunk c of row r sits at chunk c ^ f(r), with f chosen so that
// the K reads (one chunk of 8 or 16 consecutive rows), the V transpose reads
// (4 chunks of 4 consecutive rows) and the stores are all free of bank
// conflicts. Paged caches look their block-table entries up ahead of the
// requests (scalar loads for pages of 16 rows or more).
#include "attn_common.h"
#include "prefill.h"

namespace comem {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr float kLazyMax = 8.f;        // log2 of the largest probability the lazy maximum allows
constexpr float kLazyMaxProb = 256.f;  // 2^kLazyMax

// Chunk swizzle of a row (depends on its low 4 bits only).
template <int D>
__device__ inline int swizzle(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
}

enum class PLayout { kContig, kPaged, kPagedFine };

typedef __attribute__((address_space(3))) void lds_void;

// LDS byte address of a pointer into LDS (uniform: the caller's addresses are).
__device__ inline uint32_t lds_address(char* p) {
  return static_cast<uint32_t>(uniform_i32(static_cast<int>(reinterpret_cast<uintptr_t>((lds_void*)p))));
}

// Wave w loads rows 16 w .. 16 w + 15 of every K and V tile straight into
// LDS (buffer loads with an LDS destination, no registers in between).
// Instruction u writes 1 KiB from row 16 w + RPI u on: lane l the 16 bytes at
// LDS offset 16 l, i.e. physical chunk l % CH of row 16 w + RPI u + l / CH,
// which holds logical chunk (l % CH) ^ f(row). The swizzle depends on the
// row's low 4 bits only, so the lane offsets are the same for every tile and
// group. Rows past the keys a block needs are outside the descriptor and
// arrive as zeros (checked on the device); a zero V row times a zero weight
// adds nothing. Small pages (a 16-row group spanning pages) take per-lane
// addresses, with rows past the needed keys clamped to the last one.
template <int D, PLayout LAYOUT>
struct TileLoader {
  static constexpr int CH = D / 8;      // 16-byte chunks per row
  static constexpr int RPI = 64 / CH;   // rows per wave instruction (1 KiB)
  static constexpr int NI = 16 / RPI;   // instructions per 16-row group
  const char* kbase;  // K of this KV head (contiguous: at the sequence's first row)
  const char* vbase;
  const int32_t* bt_row;  // block-table row of the sequence (paged)
  int64_t stride_token;
  int64_t stride_page;
  int64_t num_pages;
  int page_shift, page_mask;
  int kend;  // keys [0, kend) are needed
  int w, lane;
  uint32_t voff[NI];     // lane offset of instruction u within a 16-row group

  __device__ void init(int wave, int ln) {
    w = wave;
    lane = ln;
#pragma unroll
    for (int u = 0; u < NI; ++u) {
      const int r = RPI * u + lane / CH;
      voff[u] = static_cast<uint32_t>(r * stride_token + 16 * ((lane % CH) ^ swizzle<D>(r)));
    }
  }

  __device__ int fine_key(int t0, int u) const { return min(t0 + 16 * w + RPI * u + lane / CH, kend - 1); }

  // A block-table entry outside the pool reads page 0.
  __device__ int32_t in_pool(int32_t page) const { return page < 0 || page >= num_pages ? 0 : page; }

  // Page lookups of one tile (K is requested two tiles ahead, V one).
  struct Pages {
    int32_t page;
    int32_t fine[NI];
  };

  // The per-group lookup reads the block table (not written during the call)
  // through the constant address space, so it becomes a scalar load. As a
  // vector load it came with a wait for every vector memory request in
  // flight, the tile requests included, in every vector stage.
  __device__ Pages pages_of(int t0) const {
    Pages pg{};
    if constexpr (LAYOUT == PLayout::kPaged) {
      typedef const __attribute__((address_space(4))) int32_t* ConstI32;
      const int g0 = t0 + 16 * w;
      pg.page = g0 < kend ? in_pool(((ConstI32)bt_row)[g0 >> page_shift]) : 0;
    } else if constexpr (LAYOUT == PLayout::kPagedFine) {
#pragma unroll
      for (int u = 0; u < NI; ++u) pg.fine[u] = in_pool(bt_row[fine_key(t0, u) >> page_shift]);
    }
    return pg;
  }

  // Tile requests, issued as inline assembly: invisible to
  // the compiler's tracking of LDS writes by vector memory, which confused
  // the tile slots at the loop's head and added waits of its own before the
  // LDS reads of the other slots. The loop orders the requests with its own
  // waits and barriers.
  //
  // A tile request: this wave's 16 rows of the K (or V) tile at key t0.
  // Contiguous and per-group paged layouts need one buffer descriptor per
  // tile; pages under 16 rows per-lane addresses.
  struct TileReq {
    u32x4 rsrc;
    const char* base;
    int t0;
    Pages pg;
  };

  __device__ TileReq tile_req(const char* base, int t0, const Pages& pg) const {
    TileReq q;
    q.base = base;
    q.t0 = t0;
    q.pg = pg;
    if constexpr (LAYOUT != PLayout::kPagedFine) {
      const int g0 = t0 + 16 * w;
      const int rows = max(0, min(kend - g0, 16));
      int64_t off;
      if constexpr (LAYOUT == PLayout::kContig) {
        off = static_cast<int64_t>(g0) * stride_token;
      } else {
        off = static_cast<int64_t>(pg.page) * stride_page + static_cast<int64_t>(g0 & page_mask) * stride_token;
      }
      // Raw buffer: base, no stride, size in bytes, CDNA config word.
      const uint64_t addr = reinterpret_cast<uint64_t>(base + off);
      const int64_t bytes = static_cast<int64_t>(rows) * stride_token;
      q.rsrc[0] = static_cast<uint32_t>(addr);
      q.rsrc[1] = static_cast<uint32_t>(addr >> 32) & 0xffffu;
      q.rsrc[2] = bytes > 0xffffffffll ? 0xffffffffu : static_cast<uint32_t>(bytes);
      q.rsrc[3] = static_cast<uint32_t>(kBufferConfig);
    }
    return q;
  }

  // Instruction u of a tile request (1 KiB of rows, u < NI) into LDS from
  // lds_rows, the LDS address of this wave's first row of the slot. The
  // LDS address goes in m0, an operand of the asm, so the compiler writes
  // m0 itself; the s_nop covers the wait state an LDS-bound load needs after
  // an m0 write.
  __device__ void issue(const TileReq& q, uint32_t lds_rows, int u) const {
    constexpr int RB = D * 2;
    const uint32_t lds = __builtin_amdgcn_readfirstlane(lds_rows + u * RPI * RB);  // uniform; m0 takes an SGPR
    if constexpr (LAYOUT == PLayout::kPagedFine) {
      const int t = fine_key(q.t0, u);
      const int64_t off = static_cast<int64_t>(q.pg.fine[u]) * stride_page + static_cast<int64_t>(t & page_mask) * stride_token +
                          16 * ((lane % CH) ^ swizzle<D>(RPI * u + lane / CH));
      asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(q.base + off), "{m0}"(lds) : "memory");
    } else {
      asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(voff[u]), "s"(q.rsrc), "{m0}"(lds)
                   : "memory");
    }
  }

  // LDS address of this wave's first row in a tile slot.
  __device__ uint32_t lds_rows(char* slot) const { return lds_address(slot + 16 * w * (D * 2)); }

};

// p0, p1 -> (hi, lo) bf16 pairs with p = hi + lo to about 2^-16 relative:
// hi keeps the upper 16 bits of each value, lo is the exact fp32 remainder
// rounded to nearest even.
__device__ inline void split_bf16(float p0, float p1, uint32_t& hi, uint32_t& lo) {
  const uint32_t b0 = __float_as_uint(p0), b1 = __float_as_uint(p1);
  hi = __builtin_amdgcn_perm(b1, b0, 0x07060302u);
  const f32x2 r = {p0 - __uint_as_float(b0 & 0xffff0000u), p1 - __uint_as_float(b1 & 0xffff0000u)};
  lo = __builtin_bit_cast(uint32_t, __builtin_convertvector(r, bf16x2));
}

// Per-lane LDS offsets, fixed for the whole kernel.
template <int D>
struct LaneOffsets {
  int k;     // K reads: row j, logical chunk h, with the row's swizzle (XOR 32 ks for step ks)
  int v[2];  // V transpose reads, step half c2: key 8 c2 + 4 h + k / 4 of the step, head_dim 4 (k % 4)
             // + 16 (group parity) of n-tile 0 (XOR 64 n for n-tile n)
};

template <int D>
__device__ inline LaneOffsets<D> lane_offsets(int lane) {
  LaneOffsets<D> o;
  const int j = lane & 31, h = lane >> 5;
  o.k = j * (D * 2) + ((h ^ swizzle<D>(j)) << 4);
  const int k16 = lane & 15, gpar = (lane >> 4) & 1;
  const int hb = 2 * (k16 & 3) * 4;  // byte offset of head_dim 4 (k % 4) within 32 head_dim entries
#pragma unroll
  for (int c2 = 0; c2 < 2; ++c2) {
    const int r = 8 * c2 + 4 * h + (k16 >> 2);
    const int byte = 32 * gpar + hb;  // within the first 64 bytes (n-tile 0)
    o.v[c2] = r * (D * 2) + (((byte >> 4) ^ swizzle<D>(r)) << 4) + (byte & 15);
  }
  return o;
}

// The work of a tile is split into a matrix-core stage
// (scores of this tile, products of the previous one) and a vector stage
// (softmax of this tile), so that the two wave groups sharing the SIMDs can
// run one stage each at the same time.
template <int D>
struct alignas(16) LdsTile {
  char b[kPrefillTileKeys * D * 2];
};

// P^T operands of the four 16-key steps of a tile, hi and lo halves.
struct PTile {
  bf16x8 hi[2][2];
  bf16x8 lo[2][2];
};

// Schedule N LDS reads and N products of a block so that the reads run A
// ahead of the products (A reads first, then product and read alternating).
template <int N, int A>
__device__ inline void pipeline_reads() {
  __builtin_amdgcn_sched_group_barrier(0x100, A, 0);
#pragma unroll
  for (int i = 0; i < N - A; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, A, 0);
}

// Reads in flight ahead of the products: K reads in the score products, V
// transpose reads in the output products (measured best of 2/4, 4/8, 6/8).
constexpr int AHEAD_K = 6, AHEAD_V = 8;

// S^T = K_tile . Q^T for the 32 rows of a wave.
template <int D>
__device__ inline void qk_scores(const char* kt, const LaneOffsets<D>& lo, const bf16x8 (&qop)[D / 16],
                                 f32x16 (&s)[2]) {
  constexpr int KS = D / 16;
  constexpr int RB = D * 2;
  s[0] = f32x16{};
  s[1] = f32x16{};
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const int off = lo.k ^ (32 * ks);
#pragma unroll
    for (int sb = 0; sb < 2; ++sb) {
      const bf16x8 kop = *reinterpret_cast<const bf16x8*>(kt + off + 32 * sb * RB);
      s[sb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop, qop[ks], s[sb], 0, 0, 0);
    }
  }
  pipeline_reads<2 * KS, AHEAD_K>();
}

// Probabilities of one tile's scores against the reference exponent mb
// (the running maximum times scale_log2), split into P^T operands; the row's
// sum goes to psum. hook(part) runs after each quarter of the exponentials
// (tile requests placed there, kept there: requests issued back to back
// stall the wave while the address unit drains them).
template <typename Hook>
__device__ inline void probs_at(const f32x16 (&s)[2], float mb, float scale_log2, float& psum, PTile& pt, Hook&& hook) {
#pragma unroll
  for (int sb = 0; sb < 2; ++sb)
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      uint32_t ph[4], pl[4];
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const float p0 = fast_exp2(__builtin_fmaf(s[sb][8 * s2 + e], scale_log2, -mb));
        const float p1 = fast_exp2(__builtin_fmaf(s[sb][8 * s2 + e + 1], scale_log2, -mb));
        psum += p0 + p1;
        split_bf16(p0, p1, ph[e >> 1], pl[e >> 1]);
      }
      pt.hi[sb][s2] = __builtin_bit_cast(bf16x8, u32x4{ph[0], ph[1], ph[2], ph[3]});
      pt.lo[sb][s2] = __builtin_bit_cast(bf16x8, u32x4{pl[0], pl[1], pl[2], pl[3]});
      __builtin_amdgcn_sched_barrier(0);
      hook(2 * sb + s2);
      __builtin_amdgcn_sched_barrier(0);
    }
}

// Online softmax of one tile's scores: causal mask (when `masked`), lazy
// maximum with rescaling of acc and l_run, probabilities split into P^T
// operands, row sums into l_run. A row that has seen no visible key yet
// keeps a maximum of -inf and zero probabilities.
//
// The probabilities are first taken against the running maximum as it is.
// Each is at most the sum a lane takes of them, so sums of at most 2^8 in
// every lane show that no probability exceeds what the lazy maximum allows,
// and they are kept. Otherwise (or with a row that has no maximum yet) the
// whole wave takes the tile's maximum, rescales where the lazy-maximum rule
// says so and takes the probabilities again, the same steps as without the
// first try. The common case so skips the maximum (32 comparisons, a
// shuffle and a vote per lane).
template <int D, typename Hook>
__device__ inline void softmax_probs(f32x16 (&s)[2], bool masked, int t0, int limit, int h, float scale_log2,
                                     float& m_run, float& l_run, f32x16 (&acc)[D / 32], PTile& pt, Hook&& hook) {
  constexpr int NT = D / 32;
  if (masked) {
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int t = t0 + 32 * sb + 8 * (r >> 2) + 4 * h + (r & 3);
        if (t > limit) s[sb][r] = -INFINITY;
      }
  }
  // The first try runs in every wave (its hook issues the tile requests).
  float psum = 0.f;
  probs_at(s, m_run == -INFINITY ? 0.f : m_run * scale_log2, scale_log2, psum, pt, hook);
  const bool redo = m_run == -INFINITY || !(psum <= kLazyMaxProb);
  if (__builtin_amdgcn_ballot_w64(redo) != 0) {
    float mt = -INFINITY;
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s[sb][r]);
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    if (__builtin_amdgcn_ballot_w64((mt - m_run) * scale_log2 > kLazyMax) != 0) {
      const float m_new = fmaxf(m_run, mt);
      float alpha = fast_exp2((m_run - m_new) * scale_log2);
      alpha = m_new == -INFINITY ? 1.f : alpha;
#pragma unroll
      for (int n = 0; n < NT; ++n) acc[n] *= alpha;
      l_run *= alpha;
      m_run = m_new;
    }
    const float mb = m_run == -INFINITY ? 0.f : m_run * scale_log2;
    psum = 0.f;
    probs_at(s, mb, scale_log2, psum, pt, [](int) {});
  }
  l_run += psum;
}

// O^T += V_tile^T . P^T.
template <int D>
__device__ inline void pv_accumulate(const char* vt, const LaneOffsets<D>& lo, const PTile& pt, f32x16 (&acc)[D / 32]) {
  constexpr int NT = D / 32;
  constexpr int RB = D * 2;
#pragma unroll
  for (int sb = 0; sb < 2; ++sb)
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      const int step = (32 * sb + 16 * s2) * RB;
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const bf16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vt + step + (lo.v[0] ^ (64 * n))));
        const bf16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vt + step + (lo.v[1] ^ (64 * n))));
        const bf16x8 vop = __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
        acc[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop, pt.hi[sb][s2], acc[n], 0, 0, 0);
        acc[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop, pt.lo[sb][s2], acc[n], 0, 0, 0);
      }
    }
  pipeline_reads<8 * NT, AHEAD_V>();
}

// s_waitcnt immediate for vmcnt(n) with the other counters left alone (gfx9 encoding).
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// Wait until at most N of this wave's vector memory requests are in flight,
// at this point of the program (nothing is scheduled across it).
template <int N>
__device__ inline void wait_vm() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(N));
  __builtin_amdgcn_sched_barrier(0);
}

// Workgroup barrier without the memory fence of __syncthreads, whose release
// half would wait for every tile request in flight. The ping-pong loop writes
// LDS only through those requests and orders them with wait_vm; each wave's
// LDS reads have returned before its products use them.
__device__ inline void stage_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Grid: (query blocks, KV heads, sequences); the kernel maps the workgroup
// id to a work item itself (see the top of the kernel).
constexpr int kXcds = 8;  // XCDs of the GPU; workgroups are dealt to them round robin

// One workgroup of 8 waves per block of 128 rows: waves 4..7 take the same
// rows as waves 0..3 over the second half of the key tiles, with their own K
// and V slots, so each SIMD holds one wave of each half. The halves run
// their tiles in ping-pong (one half's products beside the other half's
// exponentials, see the loop) and merge their softmax states through LDS at
// the end.
template <int D, PLayout LAYOUT>
__global__ __launch_bounds__(kPrefillThreads, 1) void prefill_mfma_kernel(const PrefillParams p) {
  constexpr int KS = D / 16;
  constexpr int NT = D / 32;
  constexpr bool PAGED = LAYOUT != PLayout::kContig;
  // Work item of the workgroup. Workgroups go to the XCDs in turn (linear
  // id modulo 8). When the (sequence, KV head) pairs divide evenly over the
  // XCDs, pair hb runs all its query blocks on XCD hb % 8, so the K/V tiles
  // those blocks all stream are shared in that XCD's L2. An XCD runs its
  // pairs one after the other, so that its resident workgroups work on few
  // pairs at a time, and the blocks of a pair in order of q, the block's place
  // counted from the sequence's last (heaviest) block. Otherwise the grid
  // order is kept, with q = blockIdx.x.
  int b, hk, q;
  const int pairs = gridDim.y * gridDim.z;
  if (pairs % kXcds == 0) {
    const int lin = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
    const int x = lin % kXcds, k = lin / kXcds;
    const int r = k / gridDim.x;
    q = k - r * static_cast<int>(gridDim.x);
    const int hbp = x + kXcds * r;
    b = hbp / gridDim.y;
    hk = hbp - b * static_cast<int>(gridDim.y);
  } else {
    b = blockIdx.z;
    hk = blockIdx.y;
    q = blockIdx.x;
  }
  const int TB = p.tokens_per_block;

  int L = p.ctx_lens[b];
  int M = p.q_lens[b];
  int64_t qs = p.q_start[b];
  int64_t seq0 = PAGED ? 0 : p.seq_start[b];
  asm volatile("" : "+s"(L), "+s"(M), "+s"(qs), "+s"(seq0));  // one round trip for all four
  L = min(max(L, 0), p.max_ctx);
  M = min(max(M, 0), min(L, p.max_q));
  // q counts from each sequence's last (heaviest) block of new tokens.
  const int nblk = (M + TB - 1) / TB;
  if (q >= nblk) return;
  const int i0 = (nblk - 1 - q) * TB;
  const int prefix = L - M;
  const int kend = prefix + min(M, i0 + TB);  // keys any row of this block sees
  const int ntiles = (kend + kPrefillTileKeys - 1) / kPrefillTileKeys;
  const int nfree = (prefix + i0 + 1) / kPrefillTileKeys;  // tiles visible to every row

  const int lane = threadIdx.x & 63;
  const int wv = uniform_i32(threadIdx.x >> 6);
  const int w = wv & 3;   // row group of the wave
  const int kh = wv >> 2; // key half of the wave
  const int j = lane & 31, h = lane >> 5;
  const int row = 32 * w + j;
  const int g = row / TB;
  const int i = i0 + row % TB;  // new-token index of the lane's row
  const int ic = min(i, M - 1);  // padded rows repeat the last token; never stored
  const int qh = hk * p.group + g;
  const int limit = prefix + ic;

  TileLoader<D, LAYOUT> ld;
  ld.kbase = p.k + hk * p.stride_head + seq0 * p.stride_token;
  ld.vbase = p.v + hk * p.stride_head + seq0 * p.stride_token;
  ld.bt_row = PAGED ? p.block_table + static_cast<int64_t>(b) * p.max_pages : nullptr;
  ld.stride_token = p.stride_token;
  ld.stride_page = p.stride_page;
  ld.num_pages = p.num_pages;
  ld.page_shift = p.page_shift;
  ld.page_mask = p.page_mask;
  ld.kend = kend;
  ld.init(w, lane);

  // Q^T operand: row j, head_dim 16 ks + 8 h .. + 8 (requested after the first tile).
  bf16x8 qop[KS];
  auto load_q = [&]() {
    const char* qrow = p.q + ((qs + ic) * p.num_q_heads + qh) * (D * 2);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qop[ks] = *reinterpret_cast<const bf16x8*>(qrow + 32 * ks + 16 * h);
  };
  const LaneOffsets<D> lo = lane_offsets<D>(lane);
  f32x16 acc[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) acc[n] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  // Ping-pong key halves. Half kh (waves 4 kh .. 4 kh + 3, one per SIMD)
  // takes tiles [t_first, t_first + t_count) with its own K and V slots.
  // Its work is a chain of stages M(0) V(0) M(1) ... V(c-1) M(c), with
  // M(i) the matrix-core stage (scores of tile i, products of tile i - 1)
  // and V(i) the vector stage (softmax of tile i, which also requests V of
  // tile i + 1 and K of tile i + 2). A barrier ends every stage, and half 1
  // passes one extra barrier first, so it runs one stage behind half 0:
  // while one half's waves issue products, the other half's waves on the
  // same SIMDs compute exponentials. (A barrier counts arrivals, whatever
  // instruction the waves reach it at.) Both halves pass the same number of
  // barriers, with stages past their own tiles left empty.
  // Slots: K of tile i in ks[i % 2], V of tile i in vs[i % 2], one entry
  // per half.
  __shared__ LdsTile<D> ks0[2], ks1[2], vs0[2], vs1[2];
  using Pages = typename TileLoader<D, LAYOUT>::Pages;
  const int steps = (ntiles + 1) / 2;
  const int t_first = kh * steps;
  const int t_count = max(0, min(steps, ntiles - t_first));
  constexpr int TK = kPrefillTileKeys;
  LdsTile<D>& k0 = ks0[kh];
  LdsTile<D>& k1 = ks1[kh];
  LdsTile<D>& v0 = vs0[kh];
  LdsTile<D>& v1 = vs1[kh];
  constexpr int NI = TileLoader<D, LAYOUT>::NI;
  const uint32_t lk0 = ld.lds_rows(k0.b), lk1 = ld.lds_rows(k1.b), lv0 = ld.lds_rows(v0.b), lv1 = ld.lds_rows(v1.b);
  Pages pg_v, pg_k;  // page lookups of the next V and the next K tile to request
  {
    const Pages pg0 = ld.pages_of(TK * t_first);
    const Pages pg1 = ld.pages_of(TK * (t_first + 1));
    const auto rk0 = ld.tile_req(ld.kbase, TK * t_first, pg0);
    const auto rv0 = ld.tile_req(ld.vbase, TK * t_first, pg0);
    const auto rk1 = ld.tile_req(ld.kbase, TK * (t_first + 1), pg1);
#pragma unroll
    for (int u = 0; u < NI; ++u) {
      ld.issue(rk0, lk0, u);
      ld.issue(rv0, lv0, u);
      ld.issue(rk1, lk1, u);
    }
    pg_v = pg1;
    pg_k = ld.pages_of(TK * (t_first + 2));
  }
  load_q();
  wait_vm<0>();
  __syncthreads();

  f32x16 s[2];  // scores of a tile between its M and V stages
  PTile pt;     // probabilities of a tile between its V stage and the next M stage
  auto m_stage = [&](const LdsTile<D>& kcur, const LdsTile<D>& vprev, int c) {
    if (c >= 1 && c <= t_count) pv_accumulate<D>(vprev.b, lo, pt, acc);
    if (c < t_count) qk_scores<D>(kcur.b, lo, qop, s);
  };
  // Every V stage requests two tiles (past the half's range they are
  // unused; rows past the keys arrive as zeros), so the wait at its end
  // leaves only its own requests in flight: those of the previous V stage,
  // read in the next M stage, have landed. Both target slots were last read
  // in the M stage just before.
  constexpr int kStageLoads = 2 * TileLoader<D, LAYOUT>::NI;
  auto v_stage = [&](uint32_t kslot, uint32_t vslot, int c) {
    if (c < t_count) {
      const int t = t_first + c;
      const auto rv = ld.tile_req(ld.vbase, TK * (t + 1), pg_v);
      const auto rk = ld.tile_req(ld.kbase, TK * (t + 2), pg_k);
      pg_v = pg_k;
      pg_k = ld.pages_of(TK * (t + 3));
      if constexpr (LAYOUT == PLayout::kPagedFine) {
        // Per-lane addresses: issued at once rather than held in registers.
#pragma unroll
        for (int u = 0; u < NI; ++u) {
          ld.issue(rv, vslot, u);
          ld.issue(rk, kslot, u);
        }
        softmax_probs<D>(s, t >= nfree, TK * t, limit, h, p.scale_log2, m_run, l_run, acc, pt, [](int) {});
      } else {
        // Instructions spread over the four parts of the exponentials.
        softmax_probs<D>(s, t >= nfree, TK * t, limit, h, p.scale_log2, m_run, l_run, acc, pt, [&](int part) {
#pragma unroll
          for (int u = part * NI / 4; u < (part + 1) * NI / 4; ++u) {
            ld.issue(rv, vslot, u);
            ld.issue(rk, kslot, u);
          }
        });
      }
      wait_vm<kStageLoads>();
    }
  };
  if (kh == 1) stage_barrier();
  for (int c = 0; c <= steps; c += 2) {
    m_stage(k0, v1, c);
    stage_barrier();
    if (c < steps) {
      v_stage(lk0, lv1, c);
      stage_barrier();
      m_stage(k1, v0, c + 1);
      stage_barrier();
      if (c + 1 < steps) {
        v_stage(lk1, lv0, c + 1);
        stage_barrier();
      }
    }
  }
  if (kh == 0) stage_barrier();
  l_run += __shfl_xor(l_run, 32);
  // Half 1 leaves its state in LDS, once the last requests (unused tiles)
  // have landed; half 0 merges it into its own, waves 0-1 then waves 2-3
  // (each wave's accumulators take one 16 KB slot; lane-interleaved 16-byte
  // stores and loads, free of bank conflicts).
  wait_vm<0>();
  __syncthreads();
  float* ml = reinterpret_cast<float*>(vs0[0].b);  // m then l, [w][64 lanes] each
  if (kh == 1) {
    ml[w * 64 + lane] = m_run;
    ml[256 + w * 64 + lane] = l_run;
  }
  for (int pass = 0; pass < 2; ++pass) {
    float4* st = reinterpret_cast<float4*>(ks0[w & 1].b);  // [4 NT][64 lanes]
    if (kh == 1 && (w >> 1) == pass) {
#pragma unroll
      for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4)
          st[(4 * n + r4) * 64 + lane] = make_float4(acc[n][4 * r4], acc[n][4 * r4 + 1], acc[n][4 * r4 + 2], acc[n][4 * r4 + 3]);
    }
    __syncthreads();
    if (kh == 0 && (w >> 1) == pass) {
      const float m1 = ml[w * 64 + lane];
      const float l1 = ml[256 + w * 64 + lane];
      const float mn = fmaxf(m_run, m1);  // finite: half 0 holds key 0, visible to every row
      const float a0 = fast_exp2((m_run - mn) * p.scale_log2);
      const float a1 = m1 == -INFINITY ? 0.f : fast_exp2((m1 - mn) * p.scale_log2);
#pragma unroll
      for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          const float4 o1 = st[(4 * n + r4) * 64 + lane];
          acc[n][4 * r4] = acc[n][4 * r4] * a0 + o1.x * a1;
          acc[n][4 * r4 + 1] = acc[n][4 * r4 + 1] * a0 + o1.y * a1;
          acc[n][4 * r4 + 2] = acc[n][4 * r4 + 2] * a0 + o1.z * a1;
          acc[n][4 * r4 + 3] = acc[n][4 * r4 + 3] * a0 + o1.w * a1;
        }
      l_run = l_run * a0 + l1 * a1;
      m_run = mn;
    }
    __syncthreads();
  }
  if (kh == 1) return;
  if (i >= M) return;
  const float inv = 1.f / l_run;
  const int64_t orow = (qs + i) * p.num_q_heads + qh;
  float* o = p.out + orow * D;
  // acc[n] register r holds head_dim 32 n + 8 (r / 4) + 4 h + r % 4.
#pragma unroll
  for (int n = 0; n < NT; ++n)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4)
      *reinterpret_cast<float4*>(o + 32 * n + 8 * r4 + 4 * h) =
          make_float4(acc[n][4 * r4] * inv, acc[n][4 * r4 + 1] * inv, acc[n][4 * r4 + 2] * inv,
                      acc[n][4 * r4 + 3] * inv);
  if (h == 0 && p.lse != nullptr) p.lse[orow] = (m_run * p.scale_log2 + log2f(l_run)) * kLn2;
}

// Every form the host may launch, instantiated explicitly (clang emitted the
// host launch stubs of only some of the instantiations referenced below).
#define COMEM_PREFILL_FORMS(D, L) template __global__ void prefill_mfma_kernel<D, PLayout::L>(const PrefillParams);
COMEM_PREFILL_FORMS(128, kContig)
COMEM_PREFILL_FORMS(128, kPaged)
COMEM_PREFILL_FORMS(128, kPagedFine)
COMEM_PREFILL_FORMS(64, kContig)
COMEM_PREFILL_FORMS(64, kPaged)
COMEM_PREFILL_FORMS(64, kPagedFine)
#undef COMEM_PREFILL_FORMS

}  // namespace

template <int D>
PrefillKernelFn prefill_by_layout(int page_size) {
  // page_size 0: contiguous cache. A paged cache takes the per-group path when
  // a wave's 16-row group of a tile fits in a page.
  PrefillKernelFn fn = prefill_mfma_kernel<D, PLayout::kPagedFine>;
  if (page_size == 0) fn = prefill_mfma_kernel<D, PLayout::kContig>;
  else if (page_size >= 2048 / D) fn = prefill_mfma_kernel<D, PLayout::kPaged>;
  return fn;
}

PrefillKernelFn select_prefill_kernel(int head_dim, int page_size) {
  if (head_dim == 128) return prefill_by_layout<128>(page_size);
  if (head_dim == 64) return prefill_by_layout<64>(page_size);
  return nullptr;
}

}  // namespace comem
