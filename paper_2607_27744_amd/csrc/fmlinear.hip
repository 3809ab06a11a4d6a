// GLM FM interaction fused into the operand of the GLM linear that consumes it
// (Eq. glm-fm-two-groups feeding Eq. glm-linear; Section 3.1, closure under
// composition; Section 4.1 decomposition of both).
//
//   Y^R_r = X^R_r (X^R_r)^T                                 once per request
//   Zb_r  = W_CR vec(Y^R_r) + b                              once per request
//   out_n = act(W_CC vec([X^C_n (X^R_{m_n})^T | X^C_n (X^C_n)^T]) + Zb_{m_n})
//
// As two operators the candidate interaction Y^C (F_c (F_r + F_c) values per
// candidate) is written to HBM and read back by the linear. Here it never
// leaves the registers: a workgroup takes 128 candidates of one request (four
// waves of 32, one per SIMD) and
//   1. computes each candidate field's request-candidate products
//      P_i^T = X^R_r (X^C[:, i])^T on the matrix cores, with X^R_r the shared
//      A operand of every candidate of the tile (read once per tile), and the
//      candidate-candidate Gram entries with packed bf16 dot products on the
//      VALU (each lane holds its candidate's rows);
//   2. rounds both to bf16 and turns them, with one half-wave swap, into the
//      B operands of the linear (lane: one candidate, eight consecutive
//      interaction features);
//   3. streams W_CC through a two-slot LDS ring in chunks of 64 outputs and
//      adds Zb, the activation and stores, per chunk.
// Fast shape: F_r = 32, F_c = 8, E = 128 (the interaction workload), d_out a
// multiple of 64.
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace rocs {
namespace {

constexpr int kFlBM = 128;           // candidates per workgroup (4 waves x 32)
constexpr int kFlFR = 32, kFlFC = 8, kFlE = 128;
constexpr int kFlK = kFlFC * (kFlFR + kFlFC);   // 320 interaction features
constexpr int kFlOC = 64;            // outputs per W_CC chunk
constexpr int kFlMaxD = 4096;        // the Zb row staged in LDS (16 KiB)

// acc += <a, b> over two packed bf16 pairs, written as the instruction itself
// (each operand a 32-bit register of its own).
__device__ __forceinline__ void dot2(float& acc, uint32_t a, uint32_t b) {
  asm("v_dot2c_f32_bf16 %0, %1, %2" : "+v"(acc) : "v"(a), "v"(b));
}

// Accumulator rows 8 q + 4 hh + i (q = 2 s, 2 s + 1) of one 32-row block,
// packed to bf16 and exchanged between the wave halves: afterwards lane
// (l32, hh) holds rows 16 s + 8 hh .. + 7 of its column, in order.
__device__ __forceinline__ u32x4 fl_swap(const f32x16& acc, int s) {
  const uint32_t e0 = pack_bf16x2(acc[8 * s], acc[8 * s + 1]);
  const uint32_t e1 = pack_bf16x2(acc[8 * s + 2], acc[8 * s + 3]);
  const uint32_t o0 = pack_bf16x2(acc[8 * s + 4], acc[8 * s + 5]);
  const uint32_t o1 = pack_bf16x2(acc[8 * s + 6], acc[8 * s + 7]);
  const auto s0 = __builtin_amdgcn_permlane32_swap(e0, o0, false, false);
  const auto s1 = __builtin_amdgcn_permlane32_swap(e1, o1, false, false);
  return u32x4{s0[0], s1[0], s0[1], s1[1]};
}

// Index of the Gram entry (a, b), a <= b, in the packed upper triangle.
constexpr int tri(int a, int b) { return a * kFlFC - a * (a - 1) / 2 + (b - a); }

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void glm_fm_linear_bf16(const bf16_t* __restrict__ xr, const bf16_t* __restrict__ xc,
                        const float* __restrict__ zb, const bf16_t* __restrict__ w,
                        const int32_t* __restrict__ off, int R, int D, int relu,
                        bf16_t* __restrict__ out) {
  constexpr int BM = kFlBM, FC = kFlFC, E = kFlE, K = kFlK, OC = kFlOC;
  constexpr int ROWB = 2 * K;                   // bytes of one W_CC row (640)
  constexpr int SLOT = OC * ROWB;               // one W_CC chunk (40 KiB)
  constexpr int ZBO = 2 * SLOT;                 // Zb row (fp32)
  constexpr int KS = E / 16;                    // k-steps over the embedding
  constexpr int NPAIR = FC * (FC + 1) / 2;      // Gram entries per candidate
  constexpr int NI = SLOT / 1024;               // wave-wide DMA loads per chunk
  static_assert(NI % 4 == 0, "chunk loads split over four waves");
  static_assert(ZBO + 4 * kFlMaxD <= 160 * 1024, "LDS");
  __shared__ __attribute__((aligned(1024))) char lds[ZBO + 4 * kFlMaxD];
  ROCS_LDS char* const lds3 = (ROCS_LDS char*)lds;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;

  // Request-aligned tile slots: the whole tile shares X^R_r and Zb_r.
  const int64_t t = xcd_remap(blockIdx.x, gridDim.x);
  const int r = request_of_slot(off, R, t, 1, BM);
  const int64_t n0 = (int64_t)off[r] + (t - tile_base(off, r, 1, BM)) * BM;
  const int64_t nend = off[r + 1];
  if (n0 >= nend) return;                        // idle slot
  const int rows = (int)min((int64_t)BM, nend - n0);
  const int row = 32 * wave + l32;
  const int64_t n = n0 + min(row, rows - 1);     // clamped; extra rows never stored

  const uint32_t lbase = lds_addr(lds);
  // W_CC rows 64 c .. 64 c + 63 into ring slot `slot`; LDS chunk position
  // p of row o holds global chunk p ^ ((o / 2) % 8) (within its aligned
  // group of eight, so positions stay below 40).
  auto issue_chunk = [&](int c, int slot) __attribute__((always_inline)) {
    const char* src = reinterpret_cast<const char*>(w + (int64_t)c * OC * K);
    const uint32_t dst = lbase + (uint32_t)(slot * SLOT);
#pragma unroll
    for (int j = 0; j < NI / 4; ++j) {
      const int i = wave + 4 * j, p = 64 * i + lane;
      const int o = p / 40, pos = p % 40;
      lds_dma16_sv(src, (uint32_t)(o * ROWB + 16 * (pos ^ ((o >> 1) & 7))), dst + 1024u * i);
    }
  };

  // 1. Interaction. A = X^R_r rows (lane: request field l32, dims 16 s +
  // 8 hh ..), B = candidate field rows (lane: candidate l32, same dims). The
  // candidate's whole rows are loaded at once (one memory latency per tile),
  // before the weight stream starts.
  const bf16_t* xrr = xr + (int64_t)r * kFlFR * E + (int64_t)l32 * E + 8 * hh;
  const bf16_t* xcn = xc + n * FC * E + 8 * hh;
  u32x4 xb[KS][FC];
#pragma unroll
  for (int s = 0; s < KS; ++s)
#pragma unroll
    for (int i = 0; i < FC; ++i)
      xb[s][i] = *reinterpret_cast<const u32x4*>(xcn + i * E + 16 * s);
  bf16x8 af[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) af[s] = *reinterpret_cast<const bf16x8*>(xrr + 16 * s);
  // The rows must be in before the weight stream starts (the compiler does
  // not count the stream's loads, so its own waits would include them).
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    asm volatile("" :: "v"(as_u32x4(af[s])));
#pragma unroll
    for (int i = 0; i < FC; ++i) asm volatile("" :: "v"(xb[s][i]));
  }
  {
    const char* zs = reinterpret_cast<const char*>(zb + (int64_t)r * D);
    const int pieces = D / 4;
    for (int i = wave; 64 * i < pieces; i += 4)
      lds_dma16_sv(zs, (uint32_t)(16 * min(64 * i + lane, pieces - 1)),
                   lbase + (uint32_t)ZBO + 1024u * i);
  }
  issue_chunk(0, 0);
  f32x16 p[FC];
#pragma unroll
  for (int i = 0; i < FC; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) p[i][e] = 0.f;
  float g[NPAIR];
#pragma unroll
  for (int k = 0; k < NPAIR; ++k) g[k] = 0.f;
#pragma unroll
  for (int s = 0; s < KS; ++s) {
#pragma unroll
    for (int i = 0; i < FC; ++i) p[i] = mfma32(af[s], as_bf16x8(xb[s][i]), p[i]);
    // Gram entries over this lane's 8 dims of the step.
#pragma unroll
    for (int a = 0; a < FC; ++a)
#pragma unroll
      for (int b = a; b < FC; ++b)
#pragma unroll
        for (int k = 0; k < 4; ++k) dot2(g[tri(a, b)], xb[s][a][k], xb[s][b][k]);
  }

  // 2. B operands of the linear, one per 16-feature k-step. Request-
  // candidate steps (i, s): features 40 i + 16 s + 8 hh .. of the candidate;
  // candidate-candidate step u: lane hh holds field 2 u + hh against fields
  // 0..7 (features 40 (2 u + hh) + 32 ..).
  u32x4 bop[FC][2];
#pragma unroll
  for (int i = 0; i < FC; ++i) {
    bop[i][0] = fl_swap(p[i], 0);
    bop[i][1] = fl_swap(p[i], 1);
  }
  // The two wave halves saw different dims: sum them.
#pragma unroll
  for (int k = 0; k < NPAIR; ++k) g[k] = sum_across_halves(g[k]);
  u32x4 bcc[FC / 2];
#pragma unroll
  for (int u = 0; u < FC / 2; ++u) {
    float v[8];
#pragma unroll
    for (int j = 0; j < FC; ++j) {
      const int a0 = 2 * u, a1 = 2 * u + 1;
      const float x0 = g[a0 <= j ? tri(a0, j) : tri(j, a0)];
      const float x1 = g[a1 <= j ? tri(a1, j) : tri(j, a1)];
      v[j] = hh ? x1 : x0;
    }
    bcc[u] = u32x4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                   pack_bf16x2(v[6], v[7])};
  }

  // 3. The linear, 64 outputs per chunk: out^T = W_CC chunk (A, LDS) x
  // interaction (B, registers).
  wait_vmcnt<0>();
  ring_barrier();
  const uint32_t swz = (uint32_t)((l32 >> 1) & 7);
  const float lo = relu ? 0.f : -INFINITY;
  const int nch = D / OC;
  // k-step q of 20: (i, s) = (q / 2, q % 2) for q < 16, else Gram step q - 16.
  auto chunk_of = [&](int q) __attribute__((always_inline)) {
    const int c = q < 2 * FC ? 5 * (q >> 1) + 2 * (q & 1) + hh : 5 * (2 * (q - 2 * FC) + hh) + 4;
    return (uint32_t)c;
  };
  for (int c = 0; c < nch; ++c) {
    const int slot = c & 1;
    if (c + 1 < nch) issue_chunk(c + 1, slot ^ 1);
    const uint32_t sb = (uint32_t)(slot * SLOT) + (uint32_t)(l32 * ROWB);
    f32x16 acc[2];
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[b][e] = 0.f;
    bf16x8 wf[3][2];
    auto load_w = [&](int q, int buf) __attribute__((always_inline)) {
      const uint32_t o16 = 16u * (chunk_of(q) ^ swz);
#pragma unroll
      for (int b = 0; b < 2; ++b)
        wf[buf][b] = *reinterpret_cast<const ROCS_LDS bf16x8*>(lds3 + sb + 32 * b * ROWB + o16);
    };
    load_w(0, 0);
    load_w(1, 1);
#pragma unroll
    for (int q = 0; q < 2 * FC + FC / 2; ++q) {
      if (q + 2 < 2 * FC + FC / 2) load_w(q + 2, (q + 2) % 3);
      __builtin_amdgcn_sched_barrier(0);
      const u32x4 bq = q < 2 * FC ? bop[q >> 1][q & 1] : bcc[q - 2 * FC];
#pragma unroll
      for (int b = 0; b < 2; ++b) acc[b] = mfma32(wf[q % 3][b], as_bf16x8(bq), acc[b]);
      __builtin_amdgcn_sched_barrier(0);
    }
    // Zb, activation, bf16, 16-byte stores (outputs 64 c + 32 b + 16 s + 8 hh ..).
    bf16_t* op = out + (n0 + row) * D + OC * c + 8 * hh;
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      f32x16 v = acc[b];
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const f32x4 z = *reinterpret_cast<const ROCS_LDS f32x4*>(
            lds3 + ZBO + 4 * (OC * c + 32 * b + 8 * q4 + 4 * hh));
#pragma unroll
        for (int k = 0; k < 4; ++k) v[4 * q4 + k] = fmaxf(v[4 * q4 + k] + z[k], lo);
      }
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const u32x4 o = fl_swap(v, s);
        if (row < rows) *reinterpret_cast<u32x4*>(op + 32 * b + 16 * s) = o;
      }
    }
    wait_vmcnt<0>();          // the next chunk resident (this wave's loads)
    ring_barrier();           // every wave's loads in, this slot free
  }
}

}  // namespace

bool fm_linear_fused_shape(int f_req, int f_cand, int emb, int64_t d_out) {
  return f_req == kFlFR && f_cand == kFlFC && emb == kFlE && d_out % kFlOC == 0 &&
         d_out <= kFlMaxD;
}

hipError_t launch_fm_linear(const FmLinearArgs& a, bool fused, hipStream_t s) {
  // Request side: Y^R (the interaction's request block; on the fused path the
  // interaction kernel runs with no candidate output, its candidate tiles
  // exit at once), then Zb = W_CR Y^R + b.
  InteractionArgs ia{};
  ia.x_req = a.x_req; ia.x_cand = a.x_cand; ia.cand_offsets = a.cand_offsets;
  ia.R = a.R; ia.N = a.N; ia.f_req = a.f_req; ia.f_cand = a.f_cand; ia.emb = a.emb;
  ia.bf16 = a.bf16; ia.y_req = a.y_req; ia.y_cand = fused ? nullptr : a.y_cand;
  hipError_t e = launch_interaction(ia, a.interaction_fast, s);
  if (e != hipSuccess) return e;
  LinearArgs l{};
  l.x_req = a.y_req; l.x_cand = a.y_cand; l.w_req = a.w_req; l.w_cand = a.w_cand;
  l.bias = a.bias; l.cand_offsets = a.cand_offsets;
  l.R = a.R; l.N = a.N; l.k_req = (int64_t)a.f_req * a.f_req;
  l.k_cand = (int64_t)a.f_cand * (a.f_req + a.f_cand); l.d_out = a.d_out;
  l.bf16 = a.bf16; l.relu = a.relu; l.out = a.out; l.z = a.z; l.ids = a.ids;
  if (!fused) return launch_linear(l, a.linear_fast, s);
  if (a.N == 0) return hipSuccess;
  e = launch_request_table(l, s);
  if (e != hipSuccess) return e;
  const int64_t slots = a.R + (a.N + kFlBM - 1) / kFlBM;
  if (!grid_fits(slots, 256)) return hipErrorInvalidConfiguration;
  return launch_kernel(glm_fm_linear_bf16, dim3((uint32_t)slots), dim3(256), s,
                       static_cast<const bf16_t*>(a.x_req), static_cast<const bf16_t*>(a.x_cand),
                       static_cast<const float*>(a.z), static_cast<const bf16_t*>(a.w_cand),
                       a.cand_offsets, (int)a.R, (int)a.d_out, (int)a.relu,
                       static_cast<bf16_t*>(a.out));
}

}  // namespace rocs
