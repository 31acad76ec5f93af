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
// the KV head, so every K/V tile staged in LDS serves all of them. Wave w
// owns rows 32w .. 32w + 31 and, per 64-key tile, computes
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
//     element): lane (i, h) reads those 8 V rows at head_dim NT i .. NT i +
//     NT - 1 (NT = D / 32) and n-tile n takes entry NT i + n of each, packed
//     in pairs with v_perm. Output row i of n-tile n is head_dim NT i + n.
// P is split as P = P_hi + P_lo, both bf16 (the high half truncated, the
// exact remainder rounded to nearest even), and both halves are multiplied,
// so each weight keeps about 16 significant bits: an output is off by at
// most about 2^-15 sum_t w_t |v_t| plus fp32 rounding.
//
// K and V tiles go global -> registers -> LDS, one tile ahead of the compute,
// into two LDS buffers; 16-byte chunks are XOR-swizzled by row so that the
// K reads of 32 rows and the V reads of whole rows are free of bank
// conflicts. Paged caches look their block-table entries up one tile ahead
// of the data loads.
#include "attn_common.h"
#include "prefill.h"

namespace comem {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <int D>
struct PrefillSmem {
  static constexpr int kRowBytes = D * 2;
  static constexpr int kTileBytes = kPrefillTileKeys * kRowBytes;
  char k[2][kTileBytes];
  char v[2][kTileBytes];
};

// Byte offset of 16-byte chunk c of tile row r in LDS.
template <int D>
__device__ inline int swizzled(int r, int c) {
  constexpr int CH = D / 8;
  return r * (D * 2) + ((c ^ (r & (CH - 1))) << 4);
}

// One thread's share of a K/V tile: chunk c of rows row0 + RSTEP u.
template <int D, bool PAGED>
struct TileLoader {
  static constexpr int CH = D / 8;                    // 16-byte chunks per row
  static constexpr int RSTEP = kPrefillThreads / CH;  // rows between a thread's chunks
  static constexpr int NU = kPrefillTileKeys / RSTEP;  // chunks per thread per tensor
  const char* kbase;  // K of this KV head (contiguous: at the sequence's first row)
  const char* vbase;
  const int32_t* bt_row;  // block-table row of the sequence (paged)
  int64_t stride_token;
  int64_t stride_page;
  int page_shift, page_mask;
  int kend;  // keys [0, kend) are read; later rows repeat key kend - 1
  int c, row0;
  u32x4 kreg[NU], vreg[NU];
  int32_t page[NU];

  __device__ int key(int t0, int u) const { return min(t0 + row0 + u * RSTEP, kend - 1); }

  __device__ void fetch_pages(int t0) {
    if constexpr (PAGED) {
#pragma unroll
      for (int u = 0; u < NU; ++u) page[u] = bt_row[key(t0, u) >> page_shift];
    }
  }

  __device__ void load(int t0) {
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int t = key(t0, u);
      int64_t off;
      if constexpr (PAGED) {
        off = static_cast<int64_t>(page[u]) * stride_page + static_cast<int64_t>(t & page_mask) * stride_token;
      } else {
        off = static_cast<int64_t>(t) * stride_token;
      }
      off += c * 16;
      kreg[u] = *reinterpret_cast<const u32x4*>(kbase + off);
      vreg[u] = *reinterpret_cast<const u32x4*>(vbase + off);
    }
  }

  __device__ void store(PrefillSmem<D>& sm, int buf) const {
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int off = swizzled<D>(row0 + u * RSTEP, c);
      *reinterpret_cast<u32x4*>(sm.k[buf] + off) = kreg[u];
      *reinterpret_cast<u32x4*>(sm.v[buf] + off) = vreg[u];
    }
  }
};

// NT consecutive bf16 of a V row, as read for the V^T operand.
template <int D>
struct VPiece;
template <>
struct VPiece<128> {
  u32x2 w;
  __device__ uint32_t word(int n) const { return w[n >> 1]; }
  __device__ void read(const char* tile, int r, int j) {
    w = *reinterpret_cast<const u32x2*>(tile + swizzled<128>(r, j >> 1) + ((j & 1) << 3));
  }
};
template <>
struct VPiece<64> {
  uint32_t w;
  __device__ uint32_t word(int) const { return w; }
  __device__ void read(const char* tile, int r, int j) {
    w = *reinterpret_cast<const uint32_t*>(tile + swizzled<64>(r, j >> 2) + ((j & 3) << 2));
  }
};

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// p0, p1 -> (hi, lo) bf16 pairs with p = hi + lo to about 2^-16 relative:
// hi keeps the upper 16 bits of each value, lo is the exact fp32 remainder
// rounded to nearest even.
__device__ inline void split_bf16(float p0, float p1, uint32_t& hi, uint32_t& lo) {
  const uint32_t b0 = __float_as_uint(p0), b1 = __float_as_uint(p1);
  hi = __builtin_amdgcn_perm(b1, b0, 0x07060302u);
  const f32x2 r = {p0 - __uint_as_float(b0 & 0xffff0000u), p1 - __uint_as_float(b1 & 0xffff0000u)};
  lo = __builtin_bit_cast(uint32_t, __builtin_convertvector(r, bf16x2));
}

// One 64-key tile for the 32 rows of a wave. `limit` is the last key the
// lane's row may see; MASKED is false when every key of the tile is visible
// to every row of the workgroup.
template <int D, bool MASKED>
__device__ inline void compute_tile(const PrefillSmem<D>& sm, int buf, int t0, int limit, int j,
                                    int h, const bf16x8 (&qop)[D / 16], float scale_log2, float& m_run,
                                    float& l_run, f32x16 (&acc)[D / 32]) {
  constexpr int KS = D / 16;
  constexpr int NT = D / 32;
  const char* kt = sm.k[buf];
  const char* vt = sm.v[buf];

  f32x16 s[2];
#pragma unroll
  for (int sb = 0; sb < 2; ++sb) {
    s[sb] = f32x16{};
    const int r = 32 * sb + j;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(kt + swizzled<D>(r, 2 * ks + h));
      s[sb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qop[ks], s[sb], 0, 0, 0);
    }
  }

  // Raw scores keep their order (scale > 0), so the maximum is taken on them
  // and the scale enters once, in the exponent.
  float mt = -INFINITY;
#pragma unroll
  for (int sb = 0; sb < 2; ++sb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      if constexpr (MASKED) {
        const int t = t0 + 32 * sb + 8 * (r >> 2) + 4 * h + (r & 3);
        if (t > limit) s[sb][r] = -INFINITY;
      }
      mt = fmaxf(mt, s[sb][r]);
    }
  mt = fmaxf(mt, __shfl_xor(mt, 32));
  // The first tile holds key 0, visible to every row, so m_new is finite.
  const float m_new = fmaxf(m_run, mt);
  const float alpha = fast_exp2((m_run - m_new) * scale_log2);
  if (__builtin_amdgcn_ballot_w64(alpha != 1.f) != 0) {
#pragma unroll
    for (int n = 0; n < NT; ++n) acc[n] *= alpha;
  }
  m_run = m_new;
  const float mb = m_new * scale_log2;

  float psum = 0.f;
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
      const bf16x8 pb_hi = __builtin_bit_cast(bf16x8, u32x4{ph[0], ph[1], ph[2], ph[3]});
      const bf16x8 pb_lo = __builtin_bit_cast(bf16x8, u32x4{pl[0], pl[1], pl[2], pl[3]});
      VPiece<D> vr[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) vr[e].read(vt, 32 * sb + 16 * s2 + 8 * (e >> 2) + 4 * h + (e & 3), j);
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const uint32_t sel = (n & 1) ? 0x07060302u : 0x05040100u;
        u32x4 va;
#pragma unroll
        for (int e = 0; e < 8; e += 2) va[e >> 1] = __builtin_amdgcn_perm(vr[e + 1].word(n), vr[e].word(n), sel);
        const bf16x8 vop = __builtin_bit_cast(bf16x8, va);
        acc[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop, pb_hi, acc[n], 0, 0, 0);
        acc[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop, pb_lo, acc[n], 0, 0, 0);
      }
    }
  l_run = l_run * alpha + psum;
}

// Grid: (query blocks, KV heads, sequences). Query blocks are taken in
// reverse order so that, for causal attention, the blocks with the most keys
// start first.
template <int D, bool PAGED>
__global__ __launch_bounds__(kPrefillThreads, 2) void prefill_mfma_kernel(const PrefillParams p) {
  constexpr int KS = D / 16;
  constexpr int NT = D / 32;
  __shared__ PrefillSmem<D> sm;
  const int b = blockIdx.z, hk = blockIdx.y;
  const int qb = gridDim.x - 1 - blockIdx.x;
  const int TB = p.tokens_per_block;

  int L = p.ctx_lens[b];
  int M = p.q_lens[b];
  int64_t qs = p.q_start[b];
  int64_t seq0 = PAGED ? 0 : p.seq_start[b];
  asm volatile("" : "+s"(L), "+s"(M), "+s"(qs), "+s"(seq0));  // one round trip for all four
  M = min(M, L);
  const int i0 = qb * TB;
  if (i0 >= M) return;
  const int prefix = L - M;
  const int kend = prefix + min(M, i0 + TB);  // keys any row of this block sees
  const int ntiles = (kend + kPrefillTileKeys - 1) / kPrefillTileKeys;
  const int nfree = (prefix + i0 + 1) / kPrefillTileKeys;  // tiles visible to every row

  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int j = lane & 31, h = lane >> 5;
  const int row = 32 * w + j;
  const int g = row / TB;
  const int i = i0 + row % TB;  // new-token index of the lane's row
  const int ic = min(i, M - 1);  // padded rows repeat the last token; never stored
  const int qh = hk * p.group + g;
  const int limit = prefix + ic;

  TileLoader<D, PAGED> ld;
  ld.kbase = p.k + hk * p.stride_head + seq0 * p.stride_token;
  ld.vbase = p.v + hk * p.stride_head + seq0 * p.stride_token;
  ld.bt_row = PAGED ? p.block_table + static_cast<int64_t>(b) * p.max_pages : nullptr;
  ld.stride_token = p.stride_token;
  ld.stride_page = p.stride_page;
  ld.page_shift = p.page_shift;
  ld.page_mask = p.page_mask;
  ld.kend = kend;
  ld.c = threadIdx.x % TileLoader<D, PAGED>::CH;
  ld.row0 = threadIdx.x / TileLoader<D, PAGED>::CH;

  ld.fetch_pages(0);
  ld.load(0);
  if (ntiles > 1) ld.fetch_pages(kPrefillTileKeys);

  // Q^T operand: row j, head_dim 16 ks + 8 h .. + 8.
  bf16x8 qop[KS];
  {
    const char* qrow = p.q + ((qs + ic) * p.num_q_heads + qh) * (D * 2);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qop[ks] = *reinterpret_cast<const bf16x8*>(qrow + 32 * ks + 16 * h);
  }
  f32x16 acc[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) acc[n] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  ld.store(sm, 0);
  __syncthreads();
  // Tiles every row sees whole, then the tiles that need the causal mask.
  int t = 0;
  for (; t < nfree; ++t) {
    const bool more = t + 1 < ntiles;
    if (more) {
      ld.load(kPrefillTileKeys * (t + 1));
      if (t + 2 < ntiles) ld.fetch_pages(kPrefillTileKeys * (t + 2));
    }
    compute_tile<D, false>(sm, t & 1, kPrefillTileKeys * t, limit, j, h, qop, p.scale_log2, m_run, l_run, acc);
    if (more) ld.store(sm, (t + 1) & 1);
    __syncthreads();
  }
  for (; t < ntiles; ++t) {
    const bool more = t + 1 < ntiles;
    if (more) {
      ld.load(kPrefillTileKeys * (t + 1));
      if (t + 2 < ntiles) ld.fetch_pages(kPrefillTileKeys * (t + 2));
    }
    compute_tile<D, true>(sm, t & 1, kPrefillTileKeys * t, limit, j, h, qop, p.scale_log2, m_run, l_run, acc);
    if (more) ld.store(sm, (t + 1) & 1);
    __syncthreads();
  }

  l_run += __shfl_xor(l_run, 32);
  if (i >= M) return;
  const float inv = 1.f / l_run;
  const int64_t orow = (qs + i) * p.num_q_heads + qh;
  float* o = p.out + orow * D;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int d0 = NT * (8 * (r >> 2) + 4 * h + (r & 3));
    if constexpr (NT == 4) {
      *reinterpret_cast<float4*>(o + d0) =
          make_float4(acc[0][r] * inv, acc[1][r] * inv, acc[2][r] * inv, acc[3][r] * inv);
    } else {
      *reinterpret_cast<float2*>(o + d0) = make_float2(acc[0][r] * inv, acc[1][r] * inv);
    }
  }
  if (h == 0 && p.lse != nullptr) p.lse[orow] = (m_run * p.scale_log2 + log2f(l_run)) * kLn2;
}

}  // namespace

PrefillKernelFn select_prefill_kernel(int head_dim, bool paged) {
  if (head_dim == 128) return paged ? prefill_mfma_kernel<128, true> : prefill_mfma_kernel<128, false>;
  if (head_dim == 64) return paged ? prefill_mfma_kernel<64, true> : prefill_mfma_kernel<64, false>;
  return nullptr;
}

}  // namespace comem
