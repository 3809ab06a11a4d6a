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

#include <type_traits>

namespace rocs {
namespace {

constexpr int kTileRows = 256;   // query rows per workgroup (8 waves x 32)
constexpr int kTileKeys = 64;    // history rows per K/V stage
constexpr float kLazyRescale = 8.0f;   // log2 of the largest unnormalised weight

// ---------------------------------------------------------------------------
// bf16 MFMA kernel (32x32x16 shape), head_dim D in {64, 128}.
//
// Workgroup: 8 waves x 32 query rows = one 256-row tile. With 32 rows a wave
// needs under 256 VGPRs, so two waves share each SIMD and one wave's softmax
// (VALU) overlaps the other's matrix-core work.
//
// Scores are computed transposed, S^T = K Q^T (A = K rows from LDS, B = the
// wave's query rows held in registers for the whole history), so each lane's
// accumulator holds 16 keys of one query row: the row max needs only one
// exchange between the two wave halves. O^T = V^T P^T reuses the
// probabilities straight from registers as the B operand (the order of the
// 16 keys inside one MFMA step is a fixed permutation applied to both P and
// V^T), so V is stored transposed in LDS.
//
// Online softmax in the exp2 domain, scale * log2(e) folded into one FMA.
// The running max is only moved when a stage's max exceeds it by more than
// 2^kLazyRescale, so the accumulator rescale is skipped for almost every
// stage (unnormalised weights stay below 2^8; the final division by the row
// sum is exact in the algebra). Row sums are accumulated per wave half from
// the bf16-rounded weights the PV product uses, and combined at the end.
//
// Loads never branch: history and query row indices are clamped into range,
// and the keys past the history's end are masked (weight 0) in the last,
// ragged stage only.
// ---------------------------------------------------------------------------
constexpr int kAttnWaves = 8;
constexpr int kStages = 3;       // K/V ring buffer depth in LDS

template <int D>
__global__ __launch_bounds__(64 * kAttnWaves) void dca_attn_bf16(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const bf16_t* __restrict__ v,
    const int32_t* __restrict__ cand_off, const int32_t* __restrict__ kv_off,
    bf16_t* __restrict__ out, int R, int Tq, int H, int64_t kv_stride, float scale_log2,
    int64_t slots_per_head) {
  constexpr int NT = 64 * kAttnWaves;
  constexpr int KB = kTileKeys / 32;  // 32-key blocks per stage
  constexpr int KS = D / 16;          // MFMA steps over head_dim
  constexpr int DB = D / 32;          // 32-wide output column blocks
  constexpr int PS = kTileKeys / 16;  // MFMA steps over the stage's keys
  constexpr int KROW = D + 8;         // K stage row: 16-byte pad
  constexpr int VROW = kTileKeys + 4; // V^T stage row: 8-byte pad
  constexpr int KCH = kTileKeys * D / 8 / NT;       // 16-byte K chunks per thread
  constexpr int VUNITS = (kTileKeys / 4) * (D / 8); // (4 keys x 8 dims) V units
  static_assert(KCH >= 1 && VUNITS <= NT, "staging does not tile");
  __shared__ __attribute__((aligned(16))) bf16_t lds_k[kStages][kTileKeys][KROW];
  __shared__ __attribute__((aligned(16))) bf16_t lds_v[kStages][D][VROW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
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
    for (int c = tid; c < rows * (D / 8); c += NT) {
      const int rr = c / (D / 8), dc = (c % (D / 8)) * 8;
      *reinterpret_cast<u32x4*>(oh + rr * qs + dc) = u32x4{0u, 0u, 0u, 0u};
    }
    return;
  }

  // This wave's 32 query rows as B fragments: lane holds Q[row l32][16 ks + 8 hh .. +7].
  const int wrow0 = wave * 32;
  const bool active = wrow0 < rows;
  const int qrow = min(wrow0 + l32, rows - 1);            // clamped; extra rows never stored
  bf16x8 qf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
    qf[ks] = *reinterpret_cast<const bf16x8*>(qh + qrow * qs + 16 * ks + 8 * hh);

  // K/V staging. K: chunk c -> key c / (D/8), dims (c % (D/8)) * 8.
  // V: unit u -> keys 4 (u % 16) .. +3, dims (u / 16) * 8 .. +7, written
  // transposed as eight 4-key rows. Each thread keeps pointers to its rows of
  // stage 0 and adds the stage offset; only the last stage clamps key
  // indices to L - 1.
  const bf16_t* kh = k + kv0 * kv_stride + (int64_t)h * D;
  const bf16_t* vh = v + kv0 * kv_stride + (int64_t)h * D;
  const bool has_v = tid < VUNITS;
  const int vkg = tid % 16, vdc = (tid / 16) * 8;
  const bf16_t* kp[KCH];
  int kkey[KCH];
#pragma unroll
  for (int i = 0; i < KCH; ++i) {
    const int c = tid + NT * i;
    kkey[i] = c / (D / 8);
    kp[i] = kh + (int64_t)kkey[i] * kv_stride + (c % (D / 8)) * 8;
  }
  const bf16_t* vp = vh + (int64_t)(4 * vkg) * kv_stride + vdc;
  u32x4 rk[KCH], rv[4];
  auto load_kv = [&](int base) {
    const int64_t off = (int64_t)base * kv_stride;
    if (base + kTileKeys <= L) {
#pragma unroll
      for (int i = 0; i < KCH; ++i) rk[i] = *reinterpret_cast<const u32x4*>(kp[i] + off);
      if (has_v) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          rv[e] = *reinterpret_cast<const u32x4*>(vp + off + (int64_t)e * kv_stride);
      }
    } else {
#pragma unroll
      for (int i = 0; i < KCH; ++i) {
        const int key = min(base + kkey[i], L - 1) - kkey[i];
        rk[i] = *reinterpret_cast<const u32x4*>(kp[i] + (int64_t)key * kv_stride);
      }
      if (has_v) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int key = min(base + 4 * vkg + e, L - 1) - 4 * vkg;
          rv[e] = *reinterpret_cast<const u32x4*>(vp + (int64_t)key * kv_stride);
        }
      }
    }
  };
  auto store_kv = [&](int buf) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + NT * i;
      *reinterpret_cast<u32x4*>(&lds_k[buf][kkey[i]][(c % (D / 8)) * 8]) = rk[i];
    }
    if (has_v) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        // dims vdc + 2w (low halves of the four keys) and vdc + 2w + 1 (high halves)
        const u32x2 lo = {__builtin_amdgcn_perm(rv[1][w], rv[0][w], 0x05040100u),
                          __builtin_amdgcn_perm(rv[3][w], rv[2][w], 0x05040100u)};
        const u32x2 hi = {__builtin_amdgcn_perm(rv[1][w], rv[0][w], 0x07060302u),
                          __builtin_amdgcn_perm(rv[3][w], rv[2][w], 0x07060302u)};
        *reinterpret_cast<u32x2*>(&lds_v[buf][vdc + 2 * w][4 * vkg]) = lo;
        *reinterpret_cast<u32x2*>(&lds_v[buf][vdc + 2 * w + 1][4 * vkg]) = hi;
      }
    }
  };

  float m_run = -INFINITY, l_part = 0.f;
  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) oacc[db][e] = 0.f;

  // Scores of one stage: S^T for the 64 keys in LDS buffer `buf`. Element
  // 4 qq + i of sacc[kb] is S[key 32 kb + 8 qq + 4 hh + i][row l32].
  auto qk = [&](int buf, f32x16 (&sacc)[KB]) {
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) sacc[kb][e] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(&lds_k[buf][32 * kb + l32][16 * ks + 8 * hh]);
        sacc[kb] = mfma32(a, qf[ks], sacc[kb]);
      }
      // Keep at most two steps of K fragments in flight (register budget for
      // two waves per SIMD); the other wave on the SIMD covers the latency.
      if (ks % 2 == 1) __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Softmax, first half: mask (last stage only), row max and the lazy
  // rescale of the running state.
  auto row_max = [&](f32x16 (&sacc)[KB], auto masked, int valid) {
    if constexpr (decltype(masked)::value) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (32 * kb + 8 * (e / 4) + 4 * hh + (e % 4) >= valid) sacc[kb][e] = -INFINITY;
    }
    // Row max: 32 keys per lane, then across the two wave halves.
    float mx = sacc[0][0];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sacc[kb][e]);
    mx = max_across_halves(mx) * scale_log2;
    const bool need = mx > m_run + kLazyRescale;
    if (__ballot(need) != 0) {
      const float m_new = need ? mx : m_run;
      const float alpha = exp2f(m_run - m_new);            // 0 on the first stage
      m_run = m_new;
      l_part *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db) oacc[db] *= alpha;
    }
  };

  // Softmax, second half: probabilities and the PV product against the V^T
  // in LDS buffer `buf`.
  auto exp_pv = [&](int buf, f32x16 (&sacc)[KB]) {
    // Probabilities (bf16) as B fragments of the PV product. MFMA step ps
    // covers keys 16 ps + 4 hh + {0..3} and 16 ps + 8 + 4 hh + {0..3}:
    // elements 8 (ps % 2) .. +7 of sacc[ps / 2].
    const bf16x2 ones = {(bf16_t)1.0f, (bf16_t)1.0f};
#pragma unroll
    for (int ps = 0; ps < PS; ++ps) {
      // Each packed pair is a scalar of its own: the row-sum dot2 must not
      // read its operand out of a vector register tuple (the gfx950 code
      // generator has been seen to feed the same tuple element to every dot2
      // in that form).
      uint32_t pk[4];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float s0 = sacc[ps / 2][8 * (ps % 2) + 2 * w];
        const float s1 = sacc[ps / 2][8 * (ps % 2) + 2 * w + 1];
        pk[w] = pack_bf16x2(__builtin_amdgcn_exp2f(fmaf(s0, scale_log2, -m_run)),
                            __builtin_amdgcn_exp2f(fmaf(s1, scale_log2, -m_run)));
        l_part = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pk[w]), ones, l_part,
                                                 false);
      }
      const bf16x8 pf = as_bf16x8(u32x4{pk[0], pk[1], pk[2], pk[3]});
      // O^T += V^T P^T: A lane holds V^T[32 db + l32][the same 8 keys].
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const u32x2 lo = *reinterpret_cast<const u32x2*>(&lds_v[buf][32 * db + l32][16 * ps + 4 * hh]);
        const u32x2 hi =
            *reinterpret_cast<const u32x2*>(&lds_v[buf][32 * db + l32][16 * ps + 8 + 4 * hh]);
        oacc[db] = mfma32(as_bf16x8(u32x4{lo[0], lo[1], hi[0], hi[1]}), pf, oacc[db]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Software pipeline over stages: while the matrix cores compute the scores
  // of stage t + 1, the VALU runs the softmax of stage t, then stage t's PV
  // product follows. K/V live in a 3-deep LDS ring (stages t, t + 1 and the
  // one being filled for t + 2), so one barrier per stage suffices.
  const int ntiles = (L + kTileKeys - 1) / kTileKeys;
  const int last_valid = L - (ntiles - 1) * kTileKeys;    // keys in the last stage
  load_kv(0);
  store_kv(0);
  if (ntiles > 1) {
    load_kv(kTileKeys);
    store_kv(1);
  }
  __syncthreads();
  // One pipelined step: finish the softmax bookkeeping of stage kt (scores
  // in s_cur), start the scores of stage kt + 1 into s_next on the matrix
  // cores, and let the VALU exponentiate stage kt meanwhile, then its PV.
  f32x16 s_a[KB], s_b[KB];
  auto step = [&](int kt, f32x16 (&s_cur)[KB], f32x16 (&s_next)[KB]) {
    const bool fill = kt + 2 < ntiles;
    if (fill) load_kv((kt + 2) * kTileKeys);
    if (active) {
      row_max(s_cur, std::false_type(), kTileKeys);
      qk((kt + 1) % kStages, s_next);
      exp_pv(kt % kStages, s_cur);
    }
    if (fill) store_kv((kt + 2) % kStages);
    __syncthreads();
  };
  if (active) qk(0, s_a);
  int kt = 0;
  for (; kt + 2 < ntiles; kt += 2) {        // unrolled by two: the score buffers swap roles
    step(kt, s_a, s_b);
    step(kt + 1, s_b, s_a);
  }
  if (kt + 1 < ntiles) {
    step(kt, s_a, s_b);
    if (active) {
      row_max(s_b, std::true_type(), last_valid);
      exp_pv((ntiles - 1) % kStages, s_b);
    }
  } else if (active) {
    row_max(s_a, std::true_type(), last_valid);
    exp_pv((ntiles - 1) % kStages, s_a);
  }

  if (!active) return;
  // Element 4 qq + i of oacc[db] is O[row l32][dim 32 db + 8 qq + 4 hh + i].
  const float inv = 1.0f / sum_across_halves(l_part);
  const int rr = wrow0 + l32;
  if (rr >= rows) return;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) {
      const f32x16& o = oacc[db];
      *reinterpret_cast<u32x2*>(oh + rr * qs + 32 * db + 8 * qq + 4 * hh) =
          u32x2{pack_bf16x2(o[4 * qq] * inv, o[4 * qq + 1] * inv),
                pack_bf16x2(o[4 * qq + 2] * inv, o[4 * qq + 3] * inv)};
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
  return launch_kernel(dca_attn_bf16<D>, dim3((uint32_t)grid), dim3(64 * kAttnWaves), s,
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
