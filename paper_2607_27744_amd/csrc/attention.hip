// IKBO Deep Cross Attention (Section 3.2, Eq. dca-attention; Section 4.3).
//
// Candidate n of request r = m_n attends over r's history rows
// kv_offsets[r] .. kv_offsets[r+1]-1 of the request-batched K/V. IKBO form
// (Section 4.3.1): a workgroup owns one (head, request, tile of that
// request's query rows) and streams the request's K/V through LDS once; every
// candidate row in the tile reuses it, so K/V are read once per request tile
// instead of once per candidate, and no candidate-batched copy exists.
//
// Stacking candidates: with few query tokens per candidate (one, in the
// retrieval and ranking workloads) a tile of 256 query rows is 256/T_q
// candidates of the same request, which fills the matrix cores the way one
// long query sequence would (the paper co-processes 2-4 candidates per CTA for
// the same reason, Section 4.3.2).
//
// Work order (the paper's grid reorder for L2 locality, Section 4.3.1, done
// the MI355X way): workgroup ids are renumbered so that consecutive ones run
// on the same XCD, and the work list is ordered (head, request, tile), so the
// tiles of one (request, head) run together on one XCD and share its L2.
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace rocs {
namespace {

constexpr int kTileRows = 256;   // query rows per workgroup (4 waves x 64)
constexpr int kTileKeys = 64;    // history rows per K/V stage
constexpr float kLazyRescale = 8.0f;   // log2 of the largest unnormalised weight

// ---------------------------------------------------------------------------
// bf16 MFMA kernel, head_dim D in {64, 128}.
//
// Scores are computed transposed, S^T = K Q^T (A = K rows from LDS, B = the
// wave's query rows held in registers for the whole history), so a lane's
// accumulator quads hold 4 keys of one query row: the row max needs only a
// reduction over the four 16-lane rows of the wave. O^T = V^T P^T reuses the
// probabilities straight from registers as the B operand (the key order
// inside one 32-key MFMA step is a fixed permutation applied to both P and
// V^T), so V is stored transposed in LDS.
//
// Online softmax in the exp2 domain, scale * log2(e) folded into one FMA.
// The running max is only moved when a tile's max exceeds it by more than
// 2^kLazyRescale, so the accumulator rescale is skipped for almost every tile
// (unnormalised weights stay below 2^8; the final division by the row sum is
// exact in the algebra). Row sums are accumulated per 16-lane row from the
// bf16-rounded weights the PV product uses, and reduced once at the end.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void dca_attn_bf16(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const bf16_t* __restrict__ v,
    const int32_t* __restrict__ cand_off, const int32_t* __restrict__ kv_off,
    bf16_t* __restrict__ out, int R, int Tq, int H, int64_t kv_stride, float scale_log2,
    int64_t slots_per_head) {
  constexpr int RB = 4;               // 16-row blocks per wave
  constexpr int KS = D / 32;          // MFMA steps over head_dim
  constexpr int DB = D / 16;          // 16-wide output column blocks
  constexpr int KROW = D + 8;         // K stage row: 16-byte pad
  constexpr int VROW = kTileKeys + 4; // V^T stage row: 8-byte pad
  constexpr int KCH = kTileKeys * D / 8 / 256;     // 16-byte K chunks per thread
  constexpr int VUNITS = (kTileKeys / 4) * (D / 8); // (4 keys x 8 dims) V units
  __shared__ __attribute__((aligned(16))) bf16_t lds_k[2][kTileKeys][KROW];
  __shared__ __attribute__((aligned(16))) bf16_t lds_v[2][D][VROW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, g = lane >> 4;
  const uint32_t work = xcd_remap(blockIdx.x, gridDim.x);
  const int h = (int)(work / (uint64_t)slots_per_head);
  const int64_t slot = (int64_t)(work % (uint64_t)slots_per_head);
  const int r = request_of_slot(cand_off, R, slot, Tq, kTileRows);
  const int64_t j = slot - tile_base(cand_off, r, Tq, kTileRows);
  const int64_t rend = (int64_t)cand_off[r + 1] * Tq;
  const int64_t row0 = (int64_t)cand_off[r] * Tq + j * kTileRows;
  if (row0 >= rend) return;                               // idle slot
  const int rows = (int)(rend - row0 < kTileRows ? rend - row0 : kTileRows);
  const int64_t kv0 = kv_off[r];
  const int L = kv_off[r + 1] - (int)kv0;
  const int64_t qs = (int64_t)H * D;                      // q / out row stride
  const bf16_t* qh = q + row0 * qs + (int64_t)h * D;
  bf16_t* oh = out + row0 * qs + (int64_t)h * D;

  if (L == 0) {                                           // empty history: zeros
    for (int c = tid; c < rows * (D / 8); c += 256) {
      const int rr = c / (D / 8), dc = (c % (D / 8)) * 8;
      *reinterpret_cast<u32x4*>(oh + rr * qs + dc) = u32x4{0u, 0u, 0u, 0u};
    }
    return;
  }

  // This wave's query rows, as B fragments: lane holds Q[row lr][8g .. 8g+7]
  // of each 16-row block and 32-wide head_dim step.
  const int wrow0 = wave * 64;
  const bool active = wrow0 < rows;
  bf16x8 qf[RB][KS];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int rr = wrow0 + 16 * rb + lr;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[rb][ks] = as_bf16x8(load16(qh + rr * qs + 32 * ks + 8 * g, rr < rows));
  }

  // K/V staging. K: chunk c -> key c / (D/8), dims (c % (D/8)) * 8.
  // V: unit u -> keys 4 (u % 16) .. +3, dims (u / 16) * 8 .. +7, written
  // transposed as eight 4-key rows.
  const bf16_t* kh = k + kv0 * kv_stride + (int64_t)h * D;
  const bf16_t* vh = v + kv0 * kv_stride + (int64_t)h * D;
  u32x4 rk[KCH], rv[4];
  auto load_kv = [&](int base) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + 256 * i, key = c / (D / 8), dc = (c % (D / 8)) * 8;
      rk[i] = load16(kh + (int64_t)(base + key) * kv_stride + dc, base + key < L);
    }
    if (tid < VUNITS) {
      const int kg = tid % 16, dc = (tid / 16) * 8;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int key = base + 4 * kg + e;
        rv[e] = load16(vh + (int64_t)key * kv_stride + dc, key < L);
      }
    }
  };
  auto store_kv = [&](int buf) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + 256 * i, key = c / (D / 8), dc = (c % (D / 8)) * 8;
      *reinterpret_cast<u32x4*>(&lds_k[buf][key][dc]) = rk[i];
    }
    if (tid < VUNITS) {
      const int kg = tid % 16, dc = (tid / 16) * 8;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        // dims dc + 2w (low halves) and dc + 2w + 1 (high halves)
        const u32x2 lo = {(rv[0][w] & 0xffffu) | (rv[1][w] << 16),
                          (rv[2][w] & 0xffffu) | (rv[3][w] << 16)};
        const u32x2 hi = {(rv[0][w] >> 16) | (rv[1][w] & 0xffff0000u),
                          (rv[2][w] >> 16) | (rv[3][w] & 0xffff0000u)};
        *reinterpret_cast<u32x2*>(&lds_v[buf][dc + 2 * w][4 * kg]) = lo;
        *reinterpret_cast<u32x2*>(&lds_v[buf][dc + 2 * w + 1][4 * kg]) = hi;
      }
    }
  };

  float m_run[RB], l_part[RB];
  f32x4 oacc[DB][RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    m_run[rb] = -INFINITY;
    l_part[rb] = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  const int ntiles = (L + kTileKeys - 1) / kTileKeys;
  load_kv(0);
  store_kv(0);
  __syncthreads();
  for (int kt = 0; kt < ntiles; ++kt) {
    const int cur = kt & 1;
    const int base = kt * kTileKeys;
    if (kt + 1 < ntiles) load_kv(base + kTileKeys);
    if (active) {
      // S^T: sacc[kb][rb][i] = S[key 16 kb + 4 g + i][row 16 rb + lr]
      f32x4 sacc[4][RB];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) sacc[kb][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
          const bf16x8 a =
              *reinterpret_cast<const bf16x8*>(&lds_k[cur][16 * kb + lr][32 * ks + 8 * g]);
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) sacc[kb][rb] = mfma16(a, qf[rb][ks], sacc[kb][rb]);
        }
      }
      if (base + kTileKeys > L) {                         // ragged last tile
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (base + 16 * kb + 4 * g + i >= L)
#pragma unroll
              for (int rb = 0; rb < RB; ++rb) sacc[kb][rb][i] = -INFINITY;
      }
      // Row max (lane-local over 16 keys, then over the four 16-lane rows).
      float m_new[RB];
      bool need = false;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        float mx = sacc[0][rb][0];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i) mx = fmaxf(mx, sacc[kb][rb][i]);
        mx = max_across_rows(mx) * scale_log2;
        m_new[rb] = mx > m_run[rb] + kLazyRescale ? mx : m_run[rb];
        need |= m_new[rb] != m_run[rb];
      }
      if (__ballot(need) != 0) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const float alpha = exp2f(m_run[rb] - m_new[rb]);   // 0 on the first tile
          m_run[rb] = m_new[rb];
          l_part[rb] *= alpha;
#pragma unroll
          for (int db = 0; db < DB; ++db) oacc[db][rb] *= alpha;
        }
      }
      // Probabilities (bf16) as B fragments of the PV product: 32-key step
      // ks2 uses keys 32 ks2 + 4 g + {0..3} and 32 ks2 + 16 + 4 g + {0..3}.
      bf16x8 pf[2][RB];
      const bf16x2 ones = {(bf16_t)1.0f, (bf16_t)1.0f};
#pragma unroll
      for (int ks2 = 0; ks2 < 2; ++ks2)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          u32x4 pk;
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            const f32x4 s = sacc[2 * ks2 + half][rb];
            const float mr = m_run[rb];
            const uint32_t p01 = pack_bf16x2(__builtin_amdgcn_exp2f(fmaf(s[0], scale_log2, -mr)),
                                             __builtin_amdgcn_exp2f(fmaf(s[1], scale_log2, -mr)));
            const uint32_t p23 = pack_bf16x2(__builtin_amdgcn_exp2f(fmaf(s[2], scale_log2, -mr)),
                                             __builtin_amdgcn_exp2f(fmaf(s[3], scale_log2, -mr)));
            pk[2 * half] = p01;
            pk[2 * half + 1] = p23;
            l_part[rb] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, p01), ones,
                                                         l_part[rb], false);
            l_part[rb] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, p23), ones,
                                                         l_part[rb], false);
          }
          pf[ks2][rb] = as_bf16x8(pk);
        }
      // O^T += V^T P^T: A lane holds V^T[16 db + lr][the same 8 keys].
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int ks2 = 0; ks2 < 2; ++ks2) {
          const u32x2 lo = *reinterpret_cast<const u32x2*>(&lds_v[cur][16 * db + lr][32 * ks2 + 4 * g]);
          const u32x2 hi =
              *reinterpret_cast<const u32x2*>(&lds_v[cur][16 * db + lr][32 * ks2 + 16 + 4 * g]);
          const bf16x8 a = as_bf16x8(u32x4{lo[0], lo[1], hi[0], hi[1]});
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) oacc[db][rb] = mfma16(a, pf[ks2][rb], oacc[db][rb]);
        }
    }
    if (kt + 1 < ntiles) store_kv(cur ^ 1);
    __syncthreads();
  }

  if (!active) return;
  // oacc[db][rb][i] = O[row 16 rb + lr][dim 16 db + 4 g + i]
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const float inv = 1.0f / sum_across_rows(l_part[rb]);
    const int rr = wrow0 + 16 * rb + lr;
    if (rr >= rows) continue;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const f32x4 o = oacc[db][rb] * inv;
      *reinterpret_cast<u32x2*>(oh + rr * qs + 16 * db + 4 * g) =
          u32x2{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
    }
  }
}

// ---------------------------------------------------------------------------
// General kernel: any dtype, head_dim <= 256, any stride. One wave per
// (query row, head); lanes split head_dim, keys are visited in order with an
// exact (non-lazy) online softmax in fp32.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(64) void dca_attn_generic(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const int32_t* __restrict__ cand_off, const int32_t* __restrict__ kv_off,
    T* __restrict__ out, int R, int Tq, int H, int D, int64_t kv_stride, float scale) {
  const int64_t row = blockIdx.x;
  const int h = blockIdx.y, lane = threadIdx.x;
  const int r = owner_of(cand_off, R, row / Tq);
  const int64_t a = kv_off[r];
  const int L = kv_off[r + 1] - (int)a;
  const int64_t qo = (row * H + h) * D;
  float qv[4], o[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int d = lane + 64 * e;
    qv[e] = d < D ? load_f32(q + qo + d) : 0.f;
    o[e] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int jj = 0; jj < L; ++jj) {
    const int64_t ko = (a + jj) * kv_stride + (int64_t)h * D;
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int d = lane + 64 * e;
      if (d < D) s = fmaf(qv[e], load_f32(k + ko + d), s);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    s *= scale;
    const float mn = fmaxf(m, s);
    const float alpha = expf(m - mn), p = expf(s - mn);
    l = l * alpha + p;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int d = lane + 64 * e;
      o[e] = o[e] * alpha + (d < D ? p * load_f32(v + ko + d) : 0.f);
    }
    m = mn;
  }
  const float inv = L > 0 ? 1.0f / l : 0.f;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int d = lane + 64 * e;
    if (d < D) out[qo + d] = from_f32<T>(o[e] * inv);
  }
}

template <int D>
hipError_t launch_fast(const AttentionArgs& a, hipStream_t s) {
  const int64_t slots = a.R + (a.N * a.q_len + kTileRows - 1) / kTileRows;
  const int64_t grid = slots * a.heads;
  const float scale_log2 = a.scale * 1.4426950408889634f;
  return launch_kernel(dca_attn_bf16<D>, dim3((uint32_t)grid), dim3(256), s,
                       static_cast<const bf16_t*>(a.q), static_cast<const bf16_t*>(a.k),
                       static_cast<const bf16_t*>(a.v), a.cand_offsets, a.kv_offsets,
                       static_cast<bf16_t*>(a.out), (int)a.R, a.q_len, a.heads, a.kv_stride,
                       scale_log2, slots);
}

template <typename T>
hipError_t launch_generic(const AttentionArgs& a, hipStream_t s) {
  return launch_kernel(dca_attn_generic<T>, dim3((uint32_t)(a.N * a.q_len), (uint32_t)a.heads),
                       dim3(64), s, static_cast<const T*>(a.q), static_cast<const T*>(a.k),
                       static_cast<const T*>(a.v), a.cand_offsets, a.kv_offsets,
                       static_cast<T*>(a.out), (int)a.R, a.q_len, a.heads, a.head_dim,
                       a.kv_stride, a.scale);
}

}  // namespace

hipError_t launch_attention(const AttentionArgs& a, bool fast, hipStream_t s) {
  if (fast) return a.head_dim == 128 ? launch_fast<128>(a, s) : launch_fast<64>(a, s);
  return a.bf16 ? launch_generic<bf16_t>(a, s) : launch_generic<float>(a, s);
}

}  // namespace rocs
