// Two stacked IKBO linear layers with the hidden layer kept on chip
// (Section 3.1, closure under composition; Eq. glm-linear for each layer;
// Section 4.1 decomposition of the first layer).
//
//   H_n   = act1(W1_CC X^C_n + Zb_{m_n})     Zb = W1_CR X^R + b1, once per request
//   Y^C_n = act2(W2 H_n + b2)
//
// Run as two launches of the linear kernel, H makes a round trip through HBM
// (written once, read once: 2 d_hidden bytes per candidate each way, four
// times the 2 k_cand + 2 d_out bytes the pair needs at the retrieval shape).
// Here a persistent workgroup (one per CU) walks 128-candidate tiles (four
// waves of 32, one wave per SIMD). A wave keeps its candidates' X^C rows in
// registers and walks the hidden layer in chunks of 64 units: the chunk's 64
// rows of W1_CC and 64 columns of W2 come through a two-slot LDS ring (DMA
// loads, one chunk ahead, as one stream across tiles since every tile needs
// the same weights); the wave computes its 64 x 32 block of H^T on the matrix
// cores, adds the Zb row of each candidate's request and the activation,
// rounds to bf16, and feeds it straight back as the operand of the second
// product. H never leaves the registers. During a tile's last chunk the next
// tile's X^C rows and Zb rows are loaded, so a tile starts without a wait.
//
// Matrix-core roles (32x32x16 bf16 MFMA): both products are computed
// transposed, hidden / output units on the M side and candidates on the N
// side, so that a lane's accumulator holds one candidate's runs of four
// consecutive units:
//   H^T[h][n]  = sum_k W1_CC[h][k] X^C[n][k]    A = W1 rows (LDS), B = X^C rows
//   Y^T[o][n] += sum_h W2[o][h] H[n][h]         A = W2 rows (LDS), B = H
// One half-wave swap turns the H^T accumulator layout into the B operand of
// the second product (eight consecutive hidden units per lane), and the same
// swap gives 16 contiguous output bytes per lane for the stores.
//
// Tiles cover the candidates contiguously; the Zb rows of two consecutive
// requests are staged per tile, and each candidate picks its own. A tile
// that spans more than two requests (requests of fewer than 128 candidates)
// is run once per pair of requests, storing only that pair's rows.
#include "common.h"
#include "kernels.h"
#include "launch.h"

#include <climits>

namespace rocs {
namespace {

constexpr int kMlpBM = 128;          // candidates per tile (4 waves x 32)
constexpr int kMlpHC = 64;           // hidden units per chunk
constexpr int kMlpMaxHidden = 1024;  // two Zb rows per tile, double-buffered in LDS

// Chunk position of 16-byte chunk c of an LDS row: c ^ swizzle(row). With
// 16 or more chunks per row the 16 rows read by a quarter-wave at one chunk
// land on 16 distinct 16-byte bank groups (the row stride is a multiple of
// 256 bytes); with 8 chunks per row (128-byte rows) two rows share a 256-byte
// bank span, so the row's low bit selects the half and (row / 2) % 8 the
// chunk.
template <int CPR>
__device__ __forceinline__ int mlp_swizzle(int row) {
  static_assert(CPR == 8 || CPR >= 16, "row width");
  if constexpr (CPR >= 16) return row & 15;
  else return (row >> 1) & 7;
}

// Four fp32 accumulator values of one lane (units u .. u + 3 of one
// candidate) plus an additive row, then max with `lo` (0 for ReLU, -inf for
// none: no branch), as two packed bf16 pairs.
__device__ __forceinline__ void pack4(const f32x16& acc, int q, f32x4 add, float lo,
                                      uint32_t& p0, uint32_t& p1) {
  p0 = pack_bf16x2(fmaxf(acc[4 * q] + add[0], lo), fmaxf(acc[4 * q + 1] + add[1], lo));
  p1 = pack_bf16x2(fmaxf(acc[4 * q + 2] + add[2], lo), fmaxf(acc[4 * q + 3] + add[3], lo));
}

// Accumulator rows 8 q + 4 hh + i (q = 2 s, 2 s + 1) of one 32-unit block,
// packed, exchanged between the wave halves: afterwards lane (l32, hh) holds
// units 16 s + 8 hh .. + 7 of its candidate, in order.
__device__ __forceinline__ u32x4 swap_halves(const uint32_t (&p)[4][2], int s) {
  const auto s0 = __builtin_amdgcn_permlane32_swap(p[2 * s][0], p[2 * s + 1][0], false, false);
  const auto s1 = __builtin_amdgcn_permlane32_swap(p[2 * s][1], p[2 * s + 1][1], false, false);
  return u32x4{s0[0], s1[0], s0[1], s1[1]};
}

// Owner of candidate n (the largest r < R with off[r] <= n), with the
// offsets read through the scalar cache: the search is wave-uniform.
__device__ __forceinline__ int owner_scalar(const __attribute__((address_space(4))) int32_t* off,
                                            int R, int64_t n) {
  int lo = 0, hi = R - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if ((int64_t)off[mid] <= n) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// One unit of work: tile t, pass p (the p-th pair of the tile's requests).
struct MlpItem {
  int t, p, passes;
  int64_t n0;
  int rows;
  int r0, r1;          // the pair's Zb rows
  int lo, mid, hi;     // candidates [lo, mid) belong to r0, [mid, hi) to r0 + 1
};

__device__ __forceinline__ MlpItem mlp_item(const __attribute__((address_space(4))) int32_t* off,
                                            int R, int64_t N, int t, int p) {
  MlpItem it;
  it.t = t;
  it.p = p;
  it.n0 = (int64_t)t * kMlpBM;
  it.rows = (int)min((int64_t)kMlpBM, N - it.n0);
  if (off != nullptr) {
    const int ra = owner_scalar(off, R, it.n0);
    const int rb = owner_scalar(off, R, it.n0 + it.rows - 1);
    it.passes = (rb - ra) / 2 + 1;
    it.r0 = ra + 2 * p;
    it.r1 = min(it.r0 + 1, R - 1);
    it.lo = off[it.r0];
    it.mid = off[it.r0 + 1];
    it.hi = off[min(it.r0 + 2, R)];
  } else {
    it.passes = 1;
    it.r0 = it.r1 = 0;
    it.lo = 0;
    it.mid = it.hi = INT_MAX;
  }
  return it;
}

template <int KC, int DO>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void ikbo_mlp2_bf16(const bf16_t* __restrict__ x, const bf16_t* __restrict__ w1,
                    const float* __restrict__ zb, int64_t zb_stride,
                    const bf16_t* __restrict__ w2, const float* __restrict__ b2,
                    const int32_t* __restrict__ off_g, int R, int64_t N, int DH, int relu1,
                    int relu2, bf16_t* __restrict__ out) {
  constexpr int BM = kMlpBM, HC = kMlpHC;
  constexpr int ROWB1 = 2 * KC;                 // bytes of one W1 row
  constexpr int CPR1 = ROWB1 / 16;              // its 16-byte chunks
  constexpr int ROWB2 = 2 * HC;                 // bytes of one W2 row segment (128)
  constexpr int W1B = HC * ROWB1;               // W1 part of a ring slot
  constexpr int W2B = DO * ROWB2;               // W2 part of a ring slot
  constexpr int SLOT = W1B + W2B;
  constexpr int ZBUF = 2 * 4 * kMlpMaxHidden;   // two Zb rows (fp32), one buffer
  constexpr int ZBO = 2 * SLOT;                 // Zb rows, two buffers (by item parity)
  constexpr int B2O = ZBO + 2 * ZBUF;           // b2 (fp32)
  constexpr int KS = KC / 16;                   // k-steps of the first product
  constexpr int OB = DO / 32;                   // 32-unit output blocks
  constexpr int I1 = W1B / 1024, I2 = W2B / 1024;   // wave-wide DMA loads per chunk
  static_assert(I1 % 4 == 0 && I2 % 4 == 0, "chunk loads split over four waves");
  static_assert(DO * 4 <= 1024, "b2 staging");
  static_assert(B2O + 1024 <= 160 * 1024, "LDS");
  __shared__ __attribute__((aligned(1024))) char lds[B2O + 1024];
  ROCS_LDS char* const lds3 = (ROCS_LDS char*)lds;
  // The offsets are read-only for the kernel's lifetime: scalar loads.
  const __attribute__((address_space(4))) int32_t* off =
      (const __attribute__((address_space(4))) int32_t*)off_g;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int row = 32 * wave + l32;              // this lane's candidate within the tile
  const int n_tiles = (int)((N + BM - 1) / BM);
  const int G = (int)gridDim.x;
  const uint32_t lbase = lds_addr(lds);

  // Chunk c of the weights into ring slot `slot`: W1 rows 64 c .. 64 c + 63
  // (contiguous in memory), and W2 columns 64 c .. 64 c + 63 of every output
  // row. Load i of the chunk fills 1 KiB of the slot in lane order.
  auto issue_chunk = [&](int c, int slot) __attribute__((always_inline)) {
    const uint32_t dst = lbase + (uint32_t)(slot * SLOT);
    const char* s1 = reinterpret_cast<const char*>(w1 + (int64_t)c * HC * KC);
#pragma unroll
    for (int j = 0; j < I1 / 4; ++j) {
      const int i = wave + 4 * j, p = 64 * i + lane;
      const int r = p / CPR1, pos = p % CPR1;
      lds_dma16_sv(s1, (uint32_t)(r * ROWB1 + 16 * (pos ^ mlp_swizzle<CPR1>(r))),
                   dst + 1024u * i);
    }
    const char* s2 = reinterpret_cast<const char*>(w2 + (int64_t)c * HC);
#pragma unroll
    for (int j = 0; j < I2 / 4; ++j) {
      const int i = wave + 4 * j, p = 64 * i + lane;
      const int o = p >> 3, pos = p & 7;
      lds_dma16_sv(s2, (uint32_t)(o * DH * 2 + 16 * (pos ^ mlp_swizzle<8>(o))),
                   dst + (uint32_t)W1B + 1024u * i);
    }
  };
  // The item's two Zb rows into Zb buffer `buf` (lanes past the rows repeat
  // the last piece, into the buffer's padding).
  auto issue_zb = [&](const MlpItem& it, int buf) __attribute__((always_inline)) {
    const char* zs = reinterpret_cast<const char*>(zb + (int64_t)it.r0 * zb_stride);
    const int per_row = DH / 4, pieces = 2 * per_row;
    const uint32_t r1off = (uint32_t)((int64_t)(it.r1 - it.r0) * zb_stride * 4);
    for (int i = wave; 64 * i < pieces; i += 4) {
      const int p = min(64 * i + lane, pieces - 1);
      const uint32_t src = (p < per_row ? 0u : r1off) + 16u * (uint32_t)(p % per_row);
      lds_dma16_sv(zs, src, lbase + (uint32_t)(ZBO + buf * ZBUF) + 1024u * i);
    }
  };
  auto load_x = [&](const MlpItem& it, bf16x8 (&xf)[KS]) __attribute__((always_inline)) {
    const int xrow = min(row, it.rows - 1);        // clamped; extra rows never stored
    const bf16_t* xp = x + (it.n0 + xrow) * KC + 8 * hh;
#pragma unroll
    for (int s = 0; s < KS; ++s) xf[s] = *reinterpret_cast<const bf16x8*>(xp + 16 * s);
  };

  // Prologue: the first item's Zb rows and b2 (zeros when absent), the first
  // weight chunk, and the wave's 32 candidate rows as B fragments (lane:
  // row l32, features 16 s + 8 hh ..).
  MlpItem cur = mlp_item(off, R, N, (int)blockIdx.x, 0);
  if (zb != nullptr) {
    issue_zb(cur, 0);
  } else {
    for (int i = tid; i < 2 * ZBUF / 16; i += 256)
      *reinterpret_cast<ROCS_LDS u32x4*>(lds3 + ZBO + 16 * i) = u32x4{0u, 0u, 0u, 0u};
  }
  if (b2 != nullptr) {
    if (wave == 1) lds_dma16_sv(b2, (uint32_t)(16 * min(lane, DO / 4 - 1)), lbase + (uint32_t)B2O);
  } else if (tid < DO / 4) {
    *reinterpret_cast<ROCS_LDS u32x4*>(lds3 + B2O + 16 * tid) = u32x4{0u, 0u, 0u, 0u};
  }
  issue_chunk(0, 0);
  bf16x8 xf[KS], xn[KS];
  load_x(cur, xf);
  // Make the fragments resident here: the chunk loop then has only the
  // ring's DMA loads in flight, which the compiler does not count, so it
  // places no waits of its own there.
#pragma unroll
  for (int s = 0; s < KS; ++s) asm volatile("" :: "v"(as_u32x4(xf[s])));
  wait_vmcnt<0>();
  ring_barrier();

  // Fragment addresses: row l32 of a 32-row block, chunk 2 s + hh; the
  // swizzle turns the s step into an XOR with 32 s.
  const uint32_t fa1 = (uint32_t)(l32 * ROWB1 + 16 * (hh ^ mlp_swizzle<CPR1>(l32)));
  const uint32_t fa2 = (uint32_t)(l32 * ROWB2 + 16 * (hh ^ mlp_swizzle<8>(l32)));
  const float lo1 = relu1 ? 0.f : -INFINITY, lo2 = relu2 ? 0.f : -INFINITY;
  const int nch = DH / HC;
  int slot = 0, zbuf = 0;
  while (true) {
    // The next item, found while this one computes (scalar loads).
    const bool more = cur.p + 1 < cur.passes;
    const MlpItem nxt = mlp_item(off, R, N, more ? cur.t : cur.t + G, more ? cur.p + 1 : 0);
    const bool live = nxt.t < n_tiles;
    // This lane's candidate: its request's Zb row within the buffer.
    const int64_t n = cur.n0 + row;
    const uint32_t zrow = (uint32_t)(ZBO + zbuf * ZBUF + (n >= cur.mid ? 4 * DH : 0));
    f32x16 acc2[OB];
#pragma unroll
    for (int ob = 0; ob < OB; ++ob)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc2[ob][e] = 0.f;

    for (int c = 0; c < nch; ++c) {
      const bool last = c + 1 == nch;
      if (!last || live) issue_chunk(last ? 0 : c + 1, slot ^ 1);
      if (last && live) {
        if (zb != nullptr) issue_zb(nxt, zbuf ^ 1);
        load_x(nxt, xn);
      }
      const uint32_t s1 = (uint32_t)(slot * SLOT), s2 = s1 + (uint32_t)W1B;
      // H^T of the chunk (two 32-unit blocks); W1 fragments two k-steps ahead.
      bf16x8 af[3][2];
      auto load_a = [&](int s, int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int b = 0; b < 2; ++b)
          af[buf][b] = *reinterpret_cast<const ROCS_LDS bf16x8*>(
              lds3 + s1 + 32 * b * ROWB1 + (fa1 ^ (32u * s)));
      };
      load_a(0, 0);
      load_a(1, 1);
      f32x16 acc1[2];
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc1[b][e] = 0.f;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        if (s + 2 < KS) load_a(s + 2, (s + 2) % 3);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int b = 0; b < 2; ++b) acc1[b] = mfma32(af[s % 3][b], xf[s], acc1[b]);
        __builtin_amdgcn_sched_barrier(0);
      }
      // The second product's first W2 fragments and the chunk's Zb values are
      // read while the epilogue of the first runs.
      bf16x8 wf[2][OB];
      auto load_w = [&](int s, int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int ob = 0; ob < OB; ++ob)
          wf[buf][ob] = *reinterpret_cast<const ROCS_LDS bf16x8*>(
              lds3 + s2 + 32 * ob * ROWB2 + (fa2 ^ (32u * s)));
      };
      f32x4 z[2][4];
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          z[b][q] = *reinterpret_cast<const ROCS_LDS f32x4*>(
              lds3 + zrow + 4 * (HC * c + 32 * b + 8 * q + 4 * hh));
      load_w(0, 0);
      // Zb, activation, bf16: the B operands of the second product, one per
      // 16-unit k-step (lane: candidate l32, hidden units 16 s + 8 hh ..).
      u32x4 hb[4];
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        uint32_t p[4][2];
#pragma unroll
        for (int q = 0; q < 4; ++q) pack4(acc1[b], q, z[b][q], lo1, p[q][0], p[q][1]);
        hb[2 * b] = swap_halves(p, 0);
        hb[2 * b + 1] = swap_halves(p, 1);
      }
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        if (s + 1 < 4) load_w(s + 1, (s + 1) & 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int ob = 0; ob < OB; ++ob)
          acc2[ob] = mfma32(wf[s & 1][ob], as_bf16x8(hb[s]), acc2[ob]);
        __builtin_amdgcn_sched_barrier(0);
      }
      wait_vmcnt<0>();          // the next chunk (and the next item's rows) resident
      ring_barrier();           // every wave's loads in, this slot free
      slot ^= 1;
    }

    // Epilogue: b2, activation, bf16; after the swap each lane stores 16
    // contiguous bytes (outputs 32 ob + 16 s + 8 hh ..) of its candidate,
    // if it belongs to this item's pair of requests.
    const bool store = row < cur.rows && n >= cur.lo && n < cur.hi;
    bf16_t* op = out + n * DO + 8 * hh;
#pragma unroll
    for (int ob = 0; ob < OB; ++ob) {
      uint32_t p[4][2];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x4 bb = *reinterpret_cast<const ROCS_LDS f32x4*>(
            lds3 + B2O + 4 * (32 * ob + 8 * q + 4 * hh));
        pack4(acc2[ob], q, bb, lo2, p[q][0], p[q][1]);
      }
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const u32x4 v = swap_halves(p, s);
        if (store) *reinterpret_cast<u32x4*>(op + 32 * ob + 16 * s) = v;
      }
    }
    if (!live) break;
    cur = nxt;
    zbuf ^= 1;
#pragma unroll
    for (int s = 0; s < KS; ++s) xf[s] = xn[s];
  }
}

template <int KC, int DO>
hipError_t launch_fused(const Mlp2Args& a, const float* zb, int64_t zb_stride,
                        const int32_t* off, hipStream_t s) {
  int cus = 0;
  const hipError_t e = current_cu_count(&cus);
  if (e != hipSuccess) return e;
  const int64_t tiles = (a.N + kMlpBM - 1) / kMlpBM;
  const int grid = (int)(tiles < cus ? tiles : cus);
  return launch_kernel(ikbo_mlp2_bf16<KC, DO>, dim3((uint32_t)grid), dim3(256), s,
                       static_cast<const bf16_t*>(a.x_cand),
                       static_cast<const bf16_t*>(a.w1_cand), zb, zb_stride,
                       static_cast<const bf16_t*>(a.w2), a.b2, off, (int)a.R, a.N,
                       (int)a.d_hidden, (int)a.relu1, (int)a.relu2,
                       static_cast<bf16_t*>(a.out));
}

}  // namespace

bool mlp2_fused_shape(int64_t R, int64_t k_cand, int64_t d_hidden, int64_t d_out) {
  // The second Zb row of a tile is addressed by a 32-bit byte offset from
  // the first: the request table must stay under 4 GiB.
  return (k_cand == 128 || k_cand == 256) && (d_out == 128 || d_out == 256) &&
         d_hidden >= kMlpHC && d_hidden % kMlpHC == 0 && d_hidden <= kMlpMaxHidden &&
         R * d_hidden * 4 < (int64_t(1) << 32);
}

hipError_t launch_mlp2(const Mlp2Args& a, bool fused, hipStream_t s) {
  if (a.N == 0) return hipSuccess;
  LinearArgs l1{};
  l1.x_req = a.x_req; l1.x_cand = a.x_cand; l1.w_req = a.w1_req; l1.w_cand = a.w1_cand;
  l1.bias = a.b1; l1.cand_offsets = a.cand_offsets;
  l1.R = a.R; l1.N = a.N; l1.k_req = a.k_req; l1.k_cand = a.k_cand; l1.d_out = a.d_hidden;
  l1.bf16 = a.bf16; l1.relu = a.relu1; l1.z = a.z; l1.ids = a.ids;
  if (fused) {
    // The request table Zb = X^R W1_CR^T + b1 at batch size R, then the
    // fused candidate kernel.
    const float* zb = a.b1;
    int64_t stride = 0;
    const int32_t* off = nullptr;
    if (a.k_req > 0) {
      const hipError_t e = launch_request_table(l1, s);
      if (e != hipSuccess) return e;
      zb = a.z;
      stride = a.d_hidden;
      off = a.cand_offsets;
    }
    if (a.k_cand == 256)
      return a.d_out == 256 ? launch_fused<256, 256>(a, zb, stride, off, s)
                            : launch_fused<256, 128>(a, zb, stride, off, s);
    return a.d_out == 256 ? launch_fused<128, 256>(a, zb, stride, off, s)
                          : launch_fused<128, 128>(a, zb, stride, off, s);
  }
  // Two launches of the linear kernel, H through the workspace.
  l1.out = a.h;
  hipError_t e = launch_linear(l1, a.linear_fast, s);
  if (e != hipSuccess) return e;
  LinearArgs l2{};
  l2.x_cand = a.h; l2.w_cand = a.w2; l2.bias = a.b2;
  l2.R = 1; l2.N = a.N; l2.k_cand = a.d_hidden; l2.d_out = a.d_out;
  l2.bf16 = a.bf16; l2.relu = a.relu2; l2.out = a.out;
  return launch_linear(l2, a.linear_fast, s);
}

}  // namespace rocs
