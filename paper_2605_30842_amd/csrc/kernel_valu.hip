// Vector-ALU decode-attention kernel (float32 or bf16 caches) on gfx950.
//
// One workgroup = one (split j, KV head hk, sequence b); its 4 waves take
// tiles of the split in turn. Within a wave, LPR = D / VEC consecutive lanes
// cover one K/V row with one 16-byte load each (VEC elements), so a load
// instruction reads RPL = 64 / LPR whole rows; a tile is U such loads per
// lane (RPL * U tokens). Each lane computes its slice of the G dot products,
// the slices are summed across the LPR lanes of the row with xor-shuffles,
// and every lane then runs the online softmax of its row slot and
// accumulates weight * V over its own head_dim slice. The row slots of a wave
// are merged by log-sum-exp at the end.
#include "attn_common.h"

namespace comem {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <typename T>
struct Elem;
template <>
struct Elem<float> {
  static constexpr int kVec = 4;
  __device__ static void widen(const u32x4& x, float (&f)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) f[i] = __uint_as_float(x[i]);
  }
};
struct Bf16 {};
template <>
struct Elem<Bf16> {
  static constexpr int kVec = 8;
  __device__ static void widen(const u32x4& x, float (&f)[8]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(x[i] << 16);
      f[2 * i + 1] = __uint_as_float(x[i] & 0xffff0000u);
    }
  }
};

template <typename T, int D, int G, bool PAGED>
__global__ __launch_bounds__(kThreads) void decode_valu_kernel(const AttnParams p) {
  constexpr int VEC = Elem<T>::kVec;
  constexpr int EB = 16 / VEC;    // element bytes
  constexpr int LPR = D / VEC;    // lanes per row
  constexpr int RPL = 64 / LPR;   // rows per load instruction
  constexpr int U = 4;            // loads per lane per tile
  constexpr int TT = RPL * U;     // tokens per tile
  const int j = blockIdx.x, hk = blockIdx.y, b = blockIdx.z;
  const int L = checked_len(p.ctx_lens[b], p.max_ctx, p.errors);
  const int nsplit_b = L > 0 ? 1 + (L - 1) / p.chunk : 1;
  if (j >= nsplit_b) return;
  const int t_begin = j * p.chunk;
  const int t_end = t_begin + min(L - t_begin, p.chunk);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int rho = lane / LPR, ds = lane % LPR;

  __shared__ WaveState<D> ws;

  float qf[G][VEC];
  {
    const char* q0 = p.q + (static_cast<int64_t>(b) * p.num_q_heads + hk * G) * D * EB;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const u32x4 raw = *reinterpret_cast<const u32x4*>(q0 + (h * D + ds * VEC) * EB);
      Elem<T>::widen(raw, qf[h]);
#pragma unroll
      for (int e = 0; e < VEC; ++e) qf[h][e] *= p.scale_log2;
    }
  }
  const char* kb = p.k + hk * p.stride_head;
  const char* vb = p.v + hk * p.stride_head;
  const int64_t seq0 = PAGED ? 0 : p.seq_start[b];

  float m[G], l[G], acc[G][VEC];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = -INFINITY;
    l[h] = 0.f;
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[h][e] = 0.f;
  }

  const int ntok = t_end - t_begin;
  // Fused append: the wave whose tile holds token L - 1 (and every clamped
  // read of that row) stores the new rows first (not when the length was
  // clamped: that row is not the new token's).
  if (p.new_k != nullptr && t_end == L && L > 0 && w == ((L - 1 - t_begin) / TT) % kWaves && p.ctx_lens[b] == L) {
    int64_t row;
    if constexpr (PAGED) {
      row = checked_page_row(p, p.block_table[static_cast<int64_t>(b) * p.max_pages + ((L - 1) >> p.page_shift)],
                             L - 1);
    } else {
      row = (seq0 + L - 1) * p.stride_token;
    }
    store_new_token(p, b, hk, row, D * EB / 16, lane);
  }
  for (int base = t_begin + w * TT; base < t_begin + ntok; base += kWaves * TT) {
    u32x4 kr[U], vr[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = min(base + u * RPL + rho, t_end - 1);
      const int64_t off = row_offset<PAGED>(p, b, seq0, t) + ds * 16;
      kr[u] = *reinterpret_cast<const u32x4*>(kb + off);
      vr[u] = *reinterpret_cast<const u32x4*>(vb + off);
    }
    float s[U][G];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float kf[VEC];
      Elem<T>::widen(kr[u], kf);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float a = 0.f;
#pragma unroll
        for (int e = 0; e < VEC; ++e) a += qf[h][e] * kf[e];
#pragma unroll
        for (int o = LPR / 2; o >= 1; o >>= 1) a += __shfl_xor(a, o);
        s[u][h] = (base + u * RPL + rho < t_end) ? a : -INFINITY;
      }
    }
    float vf[U][VEC];
#pragma unroll
    for (int u = 0; u < U; ++u) Elem<T>::widen(vr[u], vf[u]);
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float mt = s[0][h];
#pragma unroll
      for (int u = 1; u < U; ++u) mt = fmaxf(mt, s[u][h]);
      const float m_new = fmaxf(m[h], mt);
      if (m_new == -INFINITY) continue;  // no valid token in this row slot yet
      const float alpha = fast_exp2(m[h] - m_new);
      l[h] *= alpha;
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[h][e] *= alpha;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float pu = fast_exp2(s[u][h] - m_new);
        l[h] += pu;
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[h][e] += pu * vf[u][e];
      }
      m[h] = m_new;
    }
  }

  // Merge the RPL row slots of the wave (lanes that share ds).
#pragma unroll
  for (int o = LPR; o < 64; o <<= 1) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float mo = __shfl_xor(m[h], o);
      const float lo = __shfl_xor(l[h], o);
      const float M = fmaxf(m[h], mo);
      const float a = M == -INFINITY ? 0.f : fast_exp2(m[h] - M);
      const float ao = M == -INFINITY ? 0.f : fast_exp2(mo - M);
      l[h] = l[h] * a + lo * ao;
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const float xo = __shfl_xor(acc[h][e], o);
        acc[h][e] = acc[h][e] * a + xo * ao;
      }
      m[h] = M;
    }
  }
  if (rho == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      if (ds == 0) {
        ws.m[w][h] = m[h];
        ws.l[w][h] = l[h];
      }
#pragma unroll
      for (int e = 0; e < VEC; ++e) ws.o[w][h][ds * VEC + e] = acc[h][e];
    }
  }
  __syncthreads();
  finalize_split<D>(p, ws, b, hk, j, nsplit_b);
}

template <typename T, int D, bool PAGED>
void (*pick_group(int G))(AttnParams) {
  switch (G) {
    case 1: return decode_valu_kernel<T, D, 1, PAGED>;
    case 2: return decode_valu_kernel<T, D, 2, PAGED>;
    case 4: return decode_valu_kernel<T, D, 4, PAGED>;
    case 8: return decode_valu_kernel<T, D, 8, PAGED>;
    case 16: return decode_valu_kernel<T, D, 16, PAGED>;
    default: return nullptr;
  }
}

template <typename T>
void (*pick_dim(int D, int G, bool paged))(AttnParams) {
  if (D == 128) return paged ? pick_group<T, 128, true>(G) : pick_group<T, 128, false>(G);
  if (D == 64) return paged ? pick_group<T, 64, true>(G) : pick_group<T, 64, false>(G);
  return nullptr;
}

}  // namespace

using KernelFn = void (*)(AttnParams);

KernelFn select_valu_kernel(bool bf16, int head_dim, int group, bool paged) {
  return bf16 ? pick_dim<Bf16>(head_dim, group, paged) : pick_dim<float>(head_dim, group, paged);
}

}  // namespace comem
