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
// retrieval and ranking workloads) a tile of 128 or 256 query rows holds that
// many / T_q candidates of the same request, which fills the matrix cores the way one
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

constexpr int kTileKeys = 64;    // history rows per K/V stage
constexpr int kGroupMaxRequests = 16384;            // LDS counters of the grouping kernels
constexpr int64_t kGroupMaxHist = int64_t(1) << 20;  // per-block counts scanned by one workgroup

size_t align_up256(size_t n) { return (n + 255) & ~size_t(255); }
// Online softmax bound. A stage's weights, taken against the running max as
// it stands, are accepted as they are while their per-lane sum is at most
// 2^64. Otherwise the stage takes its row max, and the running max moves to
// it only if it lies more than kLazyRescale above the running max; either
// way every accepted weight is then at most 2^64 (it may sit just under the
// bound on all 32 keys of a lane, so an accepted per-lane stage sum is at
// most 32 * 2^64). Row sums therefore stay below L * 2^64 and outputs below
// L * 2^64 * max|v|: finite in fp32 (and in bf16, which has fp32's exponent
// range) for any history shorter than 2^60 rows.
constexpr float kLazyRescale = 64.0f;     // log2 of the largest unnormalised weight
constexpr float kWeightBound = 0x1p64f;   // per-lane stage sum accepted without a row max

// Eight packed bf16 pairs added elementwise in fp32 and rounded back (RNE).
__device__ __forceinline__ u32x4 add_bf16x8(u32x4 a, u32x4 b) {
  u32x4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float lo = __builtin_bit_cast(float, a[i] << 16) + __builtin_bit_cast(float, b[i] << 16);
    const float hi = __builtin_bit_cast(float, a[i] & 0xffff0000u) +
                     __builtin_bit_cast(float, b[i] & 0xffff0000u);
    r[i] = pack_bf16x2(lo, hi);
  }
  return r;
}

// ---------------------------------------------------------------------------
// bf16 MFMA kernel (32x32x16 shape), head_dim D in {64, 128}.
//
// Workgroup: 4 waves x 32 query rows = one 128-row tile. With 32 rows a wave
// needs under 256 VGPRs (under 168 at head_dim 64), and each workgroup's K/V
// staging fits in 64 KiB of LDS (32 KiB at head_dim 64), so two workgroups
// share a CU (three at head_dim 64): each SIMD runs one wave of each. The two
// waves are not held in step by a common barrier, so one's softmax (VALU)
// overlaps the other's matrix-core work, and one workgroup's prologue (request
// lookup, query and first K/V loads) and epilogue run while the other is in
// its main loop. (A 256-row workgroup of 8 waves, one per CU, reuses each K/V
// stage for twice the rows but leaves those fixed costs exposed: 4% slower at
// a history of 2048.)
//
// Scores are computed transposed, S^T = K Q^T (A = K rows from LDS, B = the
// wave's query rows held in registers for the whole history), so each lane's
// accumulator holds 16 keys of one query row: the row max needs only one
// exchange between the two wave halves. O^T = V^T P^T reuses the
// probabilities straight from registers as the B operand (the order of the
// 16 keys inside one MFMA step is a fixed permutation applied to both P and
// V^T).
//
// K/V staging: history rows go from HBM/L2 straight into LDS with the DMA
// form of the global load (no VGPR round trip, no LDS store instructions),
// ahead of use through two 2-slot rings in LDS, one for K and one for V (K of
// stage t + 2 and V of stage t + 1 load while stage t is processed). Rows keep
// their HBM layout in
// LDS, with the 16-byte chunks of each row XOR-swizzled by the row index so
// that both fragment reads are conflict-free; V^T fragments come out of the
// row-major V stage through the transposing LDS read (ds_read_b64_tr_b16).
//
// Online softmax in the exp2 domain, scale * log2(e) folded into one FMA.
// Weights are taken against the running max as it stands; the max (and the
// accumulator rescale) is only computed when a stage's weights could pass
// 2^kLazyRescale, which the per-lane sum of the weights detects, so after the
// first stage almost no stage needs a row max (the final division by the row
// sum is exact in the algebra). Row sums are accumulated per wave half from
// the bf16-rounded weights the PV product uses, and combined at the end.
//
// Loads never branch: history and query row indices are clamped into range,
// and the keys past the history's end are masked (weight 0) in the last,
// ragged stage only.
// ---------------------------------------------------------------------------
template <int D> constexpr int attn_waves() { return 4; }  // query rows / 32 per workgroup
// Slots per K (and per V) ring: 4 stages in LDS, 64 KiB at head_dim 128, so
// two workgroups share a CU; 32 KiB at head_dim 64, where three workgroups
// share a CU (each wave within 168 registers). (At head_dim 64 a single
// 4-slot ring holding K and V of a stage together, loaded three stages
// ahead, measured 5% slower on ranking-sized histories; three-slot K and V
// rings loaded two steps ahead need runtime slot offsets, spill at 168
// registers and ran 1.5x slower.)
constexpr int kRingSlots = 2;

// MAPPED: the candidates arrive grouped by request through a permutation
// (Section 4.3.1 with a general map m): cand_off are the offsets of the
// grouped order and grouped position p holds candidate order[p], so query
// rows are gathered and output rows scattered through `order`; everything
// else is the CSR kernel.
// QPROJ: the queries are projected in the prologue (Q = round(X W_q^T), see
// below) instead of read: `q` is then X [N, T_q, kProjIn] and `wq` is W_q
// [H D, kProjIn].
constexpr int kProjIn = 256;   // input width of the fused query projection

// Tile plan (launch_attention_plan): an int32 array. Header: mode (1 =
// sorted, 0 = use the built-in order), T (tiles over all heads), R, H, T_q,
// rows per tile; then from kPlanHeader the request ids sorted by history
// length, longest first (lengths from 2^20 - 1 on count as equal; ties by
// id), and their tile offsets P[0..R]
// (P[i+1] - P[i] = H * ceil(n_r T_q / rows per tile) for the i-th request r;
// all heads of one request are consecutive, each head's tiles in order).
// Workgroup b takes tile t of that list, in chunks of kPlanChunk consecutive
// tiles per XCD: t = ((b / 8) / C * 8 + b % 8) C + (b / 8) % C, so the chunks
// of the longest histories are spread over all XCDs first and a chunk (a
// request's tiles, sharing its K/V) stays on one L2.
constexpr int kPlanHeader = 8;
constexpr int kPlanChunk = 16;
constexpr int kAttnTileRows = 128;   // query rows per tile (4 waves x 32) at head_dim 64 and 128

// Largest g in [0, n) with P[g] <= t, given P[0] <= t and P non-decreasing;
// wave-parallel like request_of_slot. Call with every lane of the wave active.
__device__ __forceinline__ int plan_group_of(const int32_t* __restrict__ P, int n, int64_t t) {
  const int lane = (int)(threadIdx.x & 63);
  int lo = 0;
  while (n > 1) {
    const int step = (n + 63) / 64;
    const int g = lo + lane * step;
    const bool ok = g < lo + n && (int64_t)P[g] <= t;
    const uint64_t m = __ballot(ok);
    const int k = 63 - __builtin_clzll(m);
    lo += k * step;
    n = min(step, n - k * step);
  }
  return __builtin_amdgcn_readfirstlane(lo);
}

template <int D, int W, bool MAPPED, bool QPROJ>
__global__ __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(D == 64 ? 3 : 2))) void dca_attn_bf16(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const bf16_t* __restrict__ v,
    const int32_t* __restrict__ cand_off, const int32_t* __restrict__ kv_off,
    bf16_t* __restrict__ out, int R, int Tq, int H, int64_t kv_stride, float scale_log2,
    int64_t slots_per_head, const int32_t* __restrict__ order, const bf16_t* __restrict__ res,
    bf16_t* __restrict__ out_sum, const bf16_t* __restrict__ wq,
    const int32_t* __restrict__ plan) {
  constexpr int NT = 64 * W;
  constexpr int TR = 32 * W;           // query rows per tile
  static_assert(TR == kAttnTileRows, "the tile plan assumes 128-row tiles");
  constexpr int KB = kTileKeys / 32;   // 32-key blocks per stage
  constexpr int KS = D / 16;           // MFMA steps over head_dim
  constexpr int DB = D / 32;           // 32-wide output column blocks
  constexpr int PS = kTileKeys / 16;   // MFMA steps over the stage's keys
  constexpr int ROWB = 2 * D;          // bytes of one history row of one head
  constexpr int CR = D / 8;            // 16-byte chunks per row
  constexpr int STAGE = kTileKeys * ROWB;             // bytes of one K (or V) stage
  constexpr int KPI = 1024 / ROWB;                    // rows per wave-wide DMA load
  constexpr int NI = kTileKeys / (KPI * W);           // DMA loads per wave, operand, stage
  static_assert(NI >= 1 && kTileKeys % (KPI * W) == 0, "staging does not tile");
  static_assert(CR * 16 == ROWB, "layout");
  constexpr int kStages = kRingSlots;
  static_assert(kStages * STAGE <= 65536, "LDS offsets must fit the 16-bit immediate");
  __shared__ __attribute__((aligned(1024))) char lds[2 * kStages * STAGE];  // K ring, V ring
  ROCS_LDS char* const lds3 = (ROCS_LDS char*)lds;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  // This workgroup's (head, request, tile of the request): from the
  // caller's plan when it matches this launch, else the built-in order
  // (head-major slots R + ceil(N T_q / TR) per head, XCD-remapped). The
  // planned grid is rounded up to whole chunk rounds; surplus workgroups
  // exit. A plan never moves an access out of range: its request ids are
  // clamped and a tile past its request's rows is idle.
  int h, r;
  int64_t j;
  const uint32_t b = blockIdx.x;
  const int64_t n_work = slots_per_head * H;
  if (plan != nullptr && plan[0] == 1 && plan[2] == R && plan[3] == H && plan[4] == Tq &&
      plan[5] == TR) {
    const uint32_t xi = b / kNumXcd;
    const int64_t t = ((int64_t)(xi / kPlanChunk) * kNumXcd + b % kNumXcd) * kPlanChunk +
                      xi % kPlanChunk;
    if (t >= plan[1]) return;
    const int32_t* P = plan + kPlanHeader + R;
    const int g = plan_group_of(P, R, t);
    r = (int)min((uint32_t)plan[kPlanHeader + g], (uint32_t)(R - 1));
    const int p0 = P[g];
    const int per_head = (P[g + 1] - p0) / H;
    if (per_head < 1) return;
    const int off = (int)(t - p0);
    h = off / per_head;
    j = off - (int64_t)h * per_head;
    if (h >= H) return;
  } else {
    if ((int64_t)b >= n_work) return;
    const uint32_t work = xcd_remap(b, (uint32_t)n_work);
    h = (int)(work / (uint64_t)slots_per_head);
    const int64_t slot = (int64_t)(work % (uint64_t)slots_per_head);
    r = request_of_slot(cand_off, R, slot, Tq, TR);
    j = slot - tile_base(cand_off, r, Tq, TR);
  }
  const int64_t rend = (int64_t)cand_off[r + 1] * Tq;
  const int64_t row0 = (int64_t)cand_off[r] * Tq + j * TR;
  if (row0 >= rend) return;                               // idle slot
  const int rows = (int)(rend - row0 < TR ? rend - row0 : TR);
  const int64_t kv0 = kv_off[r];
  const int L = kv_off[r + 1] - (int)kv0;
  const int64_t qs = (int64_t)H * D;                      // q / out row stride
  // Query / output row of the tile's row i (i < rows): row0 + i directly,
  // or through the grouped order (grouped candidate p = row / T_q holds
  // candidate order[p]).
  auto src_row = [&](int i) -> int64_t {
    const int64_t gr = row0 + i;
    if constexpr (MAPPED) {
      const int64_t p = gr / Tq;
      return (int64_t)order[p] * Tq + (gr - p * Tq);
    } else {
      return gr;
    }
  };
  const bf16_t* qh = q + (int64_t)h * D;

  if (L == 0) {                                  // empty history: zeros (and out_sum = res)
    for (int c = tid; c < rows * (D / 8); c += NT) {
      const int rr = c / (D / 8), dc = (c % (D / 8)) * 8;
      const int64_t o = src_row(rr) * qs + (int64_t)h * D + dc;
      *reinterpret_cast<u32x4*>(out + o) = u32x4{0u, 0u, 0u, 0u};
      if (res != nullptr)
        *reinterpret_cast<u32x4*>(out_sum + o) = *reinterpret_cast<const u32x4*>(res + o);
    }
    return;
  }

  // This wave's 32 query rows as B fragments: lane holds Q[row l32][16 ks + 8 hh .. +7].
  const int wrow0 = wave * 32;
  const bool active = wrow0 < rows;
  const int qrow = min(wrow0 + l32, rows - 1);            // clamped; extra rows never stored
  bf16x8 qf[KS];
  if constexpr (!QPROJ) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[ks] = *reinterpret_cast<const bf16x8*>(qh + src_row(qrow) * qs + 16 * ks + 8 * hh);
  } else {
    // The query projection of this head, fused (the candidate side of the
    // DCA query generator): Q^T = W_q,h X^T on the matrix cores, with the
    // same operand roles and k order as the streaming GEMM, so Q is
    // bit-identical to projecting first. W_q,h (D rows of 512 bytes) is
    // staged in the K/V ring before the ring's first stage; chunk c of row
    // d sits at position c ^ (d % 16), so the 16 rows read by a quarter-wave
    // fall on distinct banks. This wave's 32 rows of X are B fragments.
    static_assert(D == 64 && 2 * kStages * STAGE >= D * kProjIn * 2, "projection staging");
    constexpr int PK = kProjIn / 16;                      // k-steps (16)
    constexpr int PRB = kProjIn * 2;                      // bytes of one W_q row (512)
    constexpr int PNI = D * PRB / 1024 / W;               // DMA loads per wave (8)
    const char* wsrc = reinterpret_cast<const char*>(wq + (int64_t)h * D * kProjIn);
    const uint32_t lb = lds_addr(lds);
#pragma unroll
    for (int i = 0; i < PNI; ++i) {
      const int blk = wave * PNI + i;                     // 1 KiB: rows 2 blk, 2 blk + 1
      const int prow = 2 * blk + (lane >> 5), pos = lane & 31;
      lds_dma16_sv(wsrc, (uint32_t)(prow * PRB + 16 * (pos ^ (prow & 15))), lb + 1024u * blk);
    }
    const bf16_t* xr = q + src_row(qrow) * kProjIn + 8 * hh;
    bf16x8 xq[PK];
#pragma unroll
    for (int s2 = 0; s2 < PK; ++s2) xq[s2] = *reinterpret_cast<const bf16x8*>(xr + 16 * s2);
    wait_vmcnt<0>();
    ring_barrier();
    f32x16 pacc[2];
#pragma unroll
    for (int s2 = 0; s2 < PK; ++s2)
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int prow = 32 * b + l32;
        const bf16x8 a = *reinterpret_cast<const ROCS_LDS bf16x8*>(
            lds3 + prow * PRB + 16 * ((2 * s2 + hh) ^ (prow & 15)));
        if (s2 == 0) {
          const f32x16 zero = {};
          pacc[b] = mfma32(a, xq[0], zero);
        } else {
          pacc[b] = mfma32(a, xq[s2], pacc[b]);
        }
      }
    // Round to bf16 and exchange halves: lane (l32, hh) then holds dims
    // 32 b + 16 jj + 8 hh .. + 7 of its row, i.e. qf[2 b + jj].
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const f32x16& pa = pacc[b];
        const uint32_t e0 = pack_bf16x2(pa[8 * jj], pa[8 * jj + 1]);
        const uint32_t e1 = pack_bf16x2(pa[8 * jj + 2], pa[8 * jj + 3]);
        const uint32_t o0 = pack_bf16x2(pa[8 * jj + 4], pa[8 * jj + 5]);
        const uint32_t o1 = pack_bf16x2(pa[8 * jj + 6], pa[8 * jj + 7]);
        const auto t0 = __builtin_amdgcn_permlane32_swap(e0, o0, false, false);
        const auto t1 = __builtin_amdgcn_permlane32_swap(e1, o1, false, false);
        qf[2 * b + jj] = as_bf16x8(u32x4{t0[0], t1[0], t0[1], t1[1]});
      }
    ring_barrier();                                       // W_q's LDS goes to the K/V ring
  }

  // DMA staging. Load i of wave w fills LDS rows KPI (NI w + i) .. +KPI-1 of
  // the stage, 16 bytes per lane in lane order: lane -> row KPI (NI w + i) +
  // lane / CR, chunk position lane % CR, so the lane fetches chunk
  // (lane % CR) ^ kv_swizzle(row) of that history row.
  const char* kbase = reinterpret_cast<const char*>(k + kv0 * kv_stride + (int64_t)h * D);
  const char* vbase = reinterpret_cast<const char*>(v + kv0 * kv_stride + (int64_t)h * D);
  const int64_t rowstride = kv_stride * 2;                // bytes
  int skey[NI];
  uint32_t schunk[NI], soff[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    skey[i] = KPI * (NI * wave + i) + lane / CR;
    schunk[i] = 16u * (uint32_t)((lane % CR) ^ kv_swizzle<D>(skey[i]));
    soff[i] = (uint32_t)(skey[i] * rowstride) + schunk[i];
  }
  const uint32_t lds_base = lds_addr(lds);
  // Stage t of one operand (K: ring 0, V: ring 1) into slot t % kStages.
  auto issue_op = [&](int t, int ring) {
    const int base = t * kTileKeys;
    const char* src = ring == 0 ? kbase : vbase;
    const uint32_t dst = lds_base + (uint32_t)((ring * kStages + t % kStages) * STAGE);
    if (base + kTileKeys <= L) {
      const char* ss = src + base * rowstride;
#pragma unroll
      for (int i = 0; i < NI; ++i) lds_dma16_sv(ss, soff[i], dst + KPI * (NI * wave + i) * ROWB);
    } else {
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int64_t o = (int64_t)min(base + skey[i], L - 1) * rowstride + schunk[i];
        lds_dma16(src + o, dst + KPI * (NI * wave + i) * ROWB);
      }
    }
  };
  auto issue = [&](int t) {
    issue_op(t, 0);
    issue_op(t, 1);
  };

  // LDS fragment addresses (bytes, stage 0). K: row 32 kb + l32, chunk
  // 2 ks + hh; the swizzle turns the ks step into an XOR with 32 ks.
  const uint32_t ka0 = (uint32_t)(l32 * ROWB + 16 * (hh ^ kv_swizzle<D>(l32)));
  // V, transposing read r of step ps: 16-lane group g = lane / 16 reads rows
  // 16 ps + 4 (g / 2) + 8 r + (lane % 16) / 4, dims 32 db + 16 (g % 2) +
  // 4 (lane % 4) .. +3; the db step is an XOR with 64 db.
  uint32_t va0[2];
#pragma unroll
  for (int rr = 0; rr < 2; ++rr) {
    const int g = lane >> 4, jl = lane & 15;
    const int key = 4 * (g >> 1) + 8 * rr + (jl >> 2);
    const int chunk0 = 2 * (g & 1) + ((jl & 3) >> 1);
    va0[rr] = (uint32_t)(kStages * STAGE + key * ROWB + 16 * (chunk0 ^ kv_swizzle<D>(key)) +
                         8 * (jl & 1));
  }

  const int ntiles = (L + kTileKeys - 1) / kTileKeys;
  const int last_valid = L - (ntiles - 1) * kTileKeys;    // keys in the last stage
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
        const bf16x8 a = *reinterpret_cast<const ROCS_LDS bf16x8*>(
            lds3 + ((ka0 ^ (32u * ks)) + buf * STAGE + kb * 32 * ROWB));
        sacc[kb] = mfma32(a, qf[ks], sacc[kb]);
      }
      // Keep at most two steps of K fragments in flight (register budget for
      // two waves per SIMD); the other wave on the SIMD covers the latency.
      if (ks % 2 == 1) __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Row max of one stage (masking the keys past the history's end in the
  // last stage) and the move of the running max: only when the stage max
  // exceeds it by more than 2^kLazyRescale (always on the first stage).
  auto row_max = [&](f32x16 (&sacc)[KB], auto masked, int valid) {
    if constexpr (decltype(masked)::value) {
      // One 16-key group at a time: issued all at once, the 32 compares would
      // hold 32 lane masks (64 scalar registers) and push values to scratch.
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (32 * kb + 8 * qq + 4 * hh + i >= valid) sacc[kb][4 * qq + i] = -INFINITY;
          __builtin_amdgcn_sched_barrier(0);
        }
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

  // Weights of MFMA step ps as packed bf16 B fragments: step ps covers keys
  // 16 ps + 4 hh + {0..3} and 16 ps + 8 + 4 hh + {0..3}, elements
  // 8 (ps % 2) .. +7 of sacc[ps / 2]. Each packed pair is a scalar of its
  // own: the row-sum dot2 must not read its operand out of a vector register
  // tuple (the gfx950 code generator has been seen to feed the same tuple
  // element to every dot2 in that form). `lst` sums the bf16-rounded weights
  // the PV product uses.
  auto exp_block = [&](const f32x16 (&sacc)[KB], int ps, uint32_t (&pk)[4], float& lst) {
    const bf16x2 ones = {(bf16_t)1.0f, (bf16_t)1.0f};
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float s0 = sacc[ps / 2][8 * (ps % 2) + 2 * w];
      const float s1 = sacc[ps / 2][8 * (ps % 2) + 2 * w + 1];
      pk[w] = pack_bf16x2(__builtin_amdgcn_exp2f(fmaf(s0, scale_log2, -m_run)),
                          __builtin_amdgcn_exp2f(fmaf(s1, scale_log2, -m_run)));
      lst = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pk[w]), ones, lst, false);
    }
  };
  // O^T += V^T P^T for step ps: the A lane holds V^T[32 db + l32][the same
  // 8 keys], read transposed out of the row-major V stage.
  auto pv_block = [&](int buf, int ps, const uint32_t (&pk)[4]) {
    const bf16x8 pf = as_bf16x8(u32x4{pk[0], pk[1], pk[2], pk[3]});
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const uint32_t off = buf * STAGE + ps * 16 * ROWB;
      const u32x2 lo = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (ROCS_LDS i16x4*)(lds3 + ((va0[0] ^ (64u * db)) + off))));
      const u32x2 hi = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (ROCS_LDS i16x4*)(lds3 + ((va0[1] ^ (64u * db)) + off))));
      oacc[db] = mfma32(as_bf16x8(u32x4{lo[0], lo[1], hi[0], hi[1]}), pf, oacc[db]);
    }
  };
  // One stage of the software pipeline: the scores of the next stage (LDS
  // buffer nbuf) on the matrix cores, interleaved step by step with the
  // weights of this stage on the VALU; then this stage's PV product. The
  // weights use the running max as it stands; their per-lane sum bounds each
  // of them, so a stage whose sum stays below 2^kLazyRescale needs no max at
  // all. Otherwise (first stage, a jump of the scores, inf or NaN) the stage
  // takes the row max and recomputes its weights.
  auto stage = [&](int nbuf, f32x16 (&snext)[KB], int buf, f32x16 (&sacc)[KB]) {
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) snext[kb][e] = 0.f;
    uint32_t pk[PS][4];
    float lst = 0.f;
#pragma unroll
    for (int ps = 0; ps < PS; ++ps) {
#pragma unroll
      for (int ks = (KS / PS) * ps; ks < (KS / PS) * (ps + 1); ++ks)
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          const bf16x8 a = *reinterpret_cast<const ROCS_LDS bf16x8*>(
              lds3 + ((ka0 ^ (32u * ks)) + nbuf * STAGE + kb * 32 * ROWB));
          snext[kb] = mfma32(a, qf[ks], snext[kb]);
        }
      exp_block(sacc, ps, pk[ps], lst);
      // head_dim 128: the compiler's own interleave of these MFMAs with the
      // next step's weights measured 1.3% faster than this fixed order.
      if constexpr (D == 64) __builtin_amdgcn_sched_barrier(0);
    }
    if (__builtin_expect(__ballot(!(lst <= kWeightBound)) != 0, 0)) {
      row_max(sacc, std::false_type(), kTileKeys);
      lst = 0.f;
#pragma unroll
      for (int ps = 0; ps < PS; ++ps) exp_block(sacc, ps, pk[ps], lst);
    }
    l_part += lst;
    // The PV products run at raised wave priority, so the SIMD's other wave
    // (of the other workgroup) fills their gaps with its own work instead of
    // delaying them (about 1% at head_dim 128).
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int ps = 0; ps < PS; ++ps) {
      pv_block(buf, ps, pk[ps]);
      __builtin_amdgcn_sched_barrier(0);
    }
    __builtin_amdgcn_s_setprio(0);
  };
  // The last (possibly ragged) stage: masked row max, weights, PV.
  auto last_stage = [&](int buf, f32x16 (&sacc)[KB]) {
    row_max(sacc, std::true_type(), last_valid);
    uint32_t pk[PS][4];
    float lst = 0.f;
#pragma unroll
    for (int ps = 0; ps < PS; ++ps) exp_block(sacc, ps, pk[ps], lst);
    l_part += lst;
#pragma unroll
    for (int ps = 0; ps < PS; ++ps) pv_block(buf, ps, pk[ps]);
  };

  // Software pipeline over stages: while the matrix cores compute the scores
  // of stage t + 1, the VALU runs the softmax of stage t, then stage t's PV
  // product follows. Meanwhile K of stage t + 2 and V of stage t + 1 are
  // loaded; one barrier per stage hands the ring slots around.
  issue(0);
  if (ntiles > 1) issue_op(1, 0);
  // Everything resident, the query fragments included: from here on the
  // only vector-memory operations in flight are the ring's DMA loads, which
  // the compiler does not track, so it adds no waits of its own in the loop.
  wait_vmcnt<0>();
  ring_barrier();
  f32x16 s_a[KB], s_b[KB];
  auto step = [&](int kt, f32x16 (&s_cur)[KB], f32x16 (&s_next)[KB]) {
    // This step reads K of stage kt + 1 and V of stage kt; their other slots
    // (K of kt, V of kt - 1) were released by the last barrier.
    if (kt + 2 < ntiles) issue_op(kt + 2, 0);
    if (kt + 1 < ntiles) issue_op(kt + 1, 1);
    if (active) stage((kt + 1) % kStages, s_next, kt % kStages, s_cur);
    wait_vmcnt<0>();                                        // K of kt + 2, V of kt + 1
    ring_barrier();
  };
  if (active) qk(0, s_a);
  // Step 0 reloads K slot 0, which qk(0) has just read.
  ring_barrier();
  int kt = 0;
  for (; kt + 2 < ntiles; kt += 2) {        // unrolled by two: the score buffers swap roles
    step(kt, s_a, s_b);
    step(kt + 1, s_b, s_a);
  }
  if (kt + 1 < ntiles) {
    step(kt, s_a, s_b);
    if (active) {                              // one call site for the last stage
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) s_a[kb] = s_b[kb];
    }
  }
  if (active) last_stage((ntiles - 1) % kStages, s_a);

  // Epilogue through LDS. Once every wave is past its last stage the K/V
  // ring is idle; each wave writes its 32 normalised output rows there
  // (16 contiguous bytes per lane after a half-wave swap, row-swizzled) and
  // reads them back row-contiguous, so each store instruction covers whole
  // 2D-byte row segments instead of 16 bytes of 32 different rows.
  ring_barrier();
  if (!active) return;
  // The epilogue's addresses come from a laundered copy of the lane index:
  // derived from `lane` directly, the compiler computes them at the start
  // and holds them through the main loop, where the registers are short.
  int lane_e = lane;
  asm volatile("" : "+v"(lane_e));
  const int l32e = lane_e & 31, hhe = lane_e >> 5;
  // Element 4 qq + i of oacc[db] is O[row l32][dim 32 db + 8 qq + 4 hh + i];
  // after the swap lane (l32, hh) holds dims 32 db + 16 j + 8 hh .. +7
  // (16-byte chunk 4 db + 2 j + hh of the row).
  const float inv = 1.0f / sum_across_halves(l_part);
  const uint32_t obase = (uint32_t)(wave * 32 * ROWB);
  auto out_swz = [](int row) { return CR == 16 ? (row & 15) : ((row >> 1) & 7); };
  // Read-back layout: store instruction i covers rows RPS i .. RPS i + RPS - 1
  // of the wave's 32, lane -> row RPS i + lane / CR, chunk lane % CR. With a
  // residual, its matching 16-byte pieces are loaded first, so their latency
  // runs under the LDS round trip and no load waits behind an output store.
  constexpr int RPS = 1024 / ROWB;            // output rows per store instruction
  constexpr int NST = 32 / RPS;
  auto out_off = [&](int i) -> int64_t {
    const int row = RPS * i + lane_e / CR;
    return src_row(min(wrow0 + row, rows - 1)) * qs + (int64_t)h * D + 8 * (lane_e % CR);
  };
  u32x4 rv[NST];
  if (res != nullptr) {
#pragma unroll
    for (int i = 0; i < NST; ++i) rv[i] = *reinterpret_cast<const u32x4*>(res + out_off(i));
  }
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const f32x16& o = oacc[db];
      const uint32_t e0 = pack_bf16x2(o[8 * j] * inv, o[8 * j + 1] * inv);
      const uint32_t e1 = pack_bf16x2(o[8 * j + 2] * inv, o[8 * j + 3] * inv);
      const uint32_t o0 = pack_bf16x2(o[8 * j + 4] * inv, o[8 * j + 5] * inv);
      const uint32_t o1 = pack_bf16x2(o[8 * j + 6] * inv, o[8 * j + 7] * inv);
      const auto s0 = __builtin_amdgcn_permlane32_swap(e0, o0, false, false);
      const auto s1 = __builtin_amdgcn_permlane32_swap(e1, o1, false, false);
      const int chunk = (4 * db + 2 * j + hhe) ^ out_swz(l32e);
      *reinterpret_cast<ROCS_LDS u32x4*>(lds3 + obase + l32e * ROWB + 16 * chunk) =
          u32x4{s0[0], s1[0], s0[1], s1[1]};
    }
#pragma unroll
  for (int i = 0; i < NST; ++i) {
    const int row = RPS * i + lane_e / CR;
    const u32x4 v = *reinterpret_cast<const ROCS_LDS u32x4*>(
        lds3 + obase + row * ROWB + 16 * ((lane_e % CR) ^ out_swz(row)));
    if (wrow0 + row < rows) {
      const int64_t o = out_off(i);
      *reinterpret_cast<u32x4*>(out + o) = v;
      if (res != nullptr) *reinterpret_cast<u32x4*>(out_sum + o) = add_bf16x8(v, rv[i]);
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
    T* __restrict__ out, int R, int Tq, int H, int D, int64_t kv_stride, float scale,
    const int32_t* __restrict__ ids, const T* __restrict__ res, T* __restrict__ out_sum,
    const T* __restrict__ wq, int d_in) {
  const int64_t row = blockIdx.x;
  const int h = blockIdx.y, lane = threadIdx.x;
  // The request: from the caller's per-candidate map (clamped into [0, R),
  // so a malformed map gives wrong rows, never an access outside the
  // offsets), else from the CSR offsets.
  const int r = ids != nullptr ? (int)min((uint32_t)ids[row / Tq], (uint32_t)(R - 1))
                               : owner_of(cand_off, R, row / Tq);
  const int64_t a = kv_off[r];
  const int L = kv_off[r + 1] - (int)a;
  const int64_t qo = (row * H + h) * D;
  float qv[4], o[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int d = lane + 64 * e;
    if (wq == nullptr) {
      qv[e] = d < D ? load_f32(q + qo + d) : 0.f;
    } else if (d < D) {
      // The fused query projection: q = x W_q^T for this head's dims,
      // rounded to T as a separate projection would store it.
      const T* xr = q + row * d_in;
      const T* wr = wq + ((int64_t)h * D + d) * d_in;
      float acc = 0.f;
      for (int kk = 0; kk < d_in; ++kk) acc = fmaf(load_f32(xr + kk), load_f32(wr + kk), acc);
      const T qt = from_f32<T>(acc);
      qv[e] = load_f32(&qt);
    } else {
      qv[e] = 0.f;
    }
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
    if (d < D) {
      const T y = from_f32<T>(o[e] * inv);
      out[qo + d] = y;
      if (res != nullptr) out_sum[qo + d] = from_f32<T>(load_f32(&y) + load_f32(res + qo + d));
    }
  }
}

// ---------------------------------------------------------------------------
// Grouping a per-candidate request map by request, a stable counting sort,
// so that the tiled kernel also serves a general map (Section 4.3.1: resolve
// m_i, then share the request's K/V). order[p] lists request 0's candidates
// first, then request 1's, ..., each request's candidates in their original
// order; grp_off[R + 1] are the CSR offsets of that order. The candidates
// are cut into nb blocks of G; hist[r * nb + b] counts request r in block b,
// and its exclusive scan in that (request-major) order is the grouped
// position of request r's first candidate in block b. Ids outside [0, R)
// are clamped into range, as the other kernels do.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int clamp_request(int32_t m, int R) {
  return (int)min((uint32_t)m, (uint32_t)(R - 1));
}

__global__ __launch_bounds__(256) void group_count(const int32_t* __restrict__ ids, int64_t N,
                                                   int R, int64_t G, int nb,
                                                   int32_t* __restrict__ hist) {
  __shared__ int cnt[kGroupMaxRequests];
  const int b = blockIdx.x;
  for (int r = threadIdx.x; r < R; r += 256) cnt[r] = 0;
  __syncthreads();
  const int64_t lo = (int64_t)b * G, hi = min(lo + G, N);
  for (int64_t i = lo + threadIdx.x; i < hi; i += 256) atomicAdd(&cnt[clamp_request(ids[i], R)], 1);
  __syncthreads();
  for (int r = threadIdx.x; r < R; r += 256) hist[(int64_t)r * nb + b] = cnt[r];
}

// One workgroup: exclusive scan of hist[0 .. total) in place (each thread
// owns a contiguous run; the run sums are scanned in LDS), then the grouped
// offsets grp_off[r] = scan[r * nb], grp_off[R] = N.
__global__ __launch_bounds__(1024) void group_scan(int32_t* __restrict__ hist, int64_t total,
                                                   int R, int nb, int64_t N,
                                                   int32_t* __restrict__ grp_off) {
  __shared__ int part[1024];
  const int t = threadIdx.x;
  const int64_t per = (total + 1023) / 1024;
  const int64_t lo = min((int64_t)t * per, total), hi = min(lo + per, total);
  int sum = 0;
  for (int64_t i = lo; i < hi; ++i) sum += hist[i];
  part[t] = sum;
  __syncthreads();
  for (int d = 1; d < 1024; d <<= 1) {                    // inclusive scan of the run sums
    const int add = t >= d ? part[t - d] : 0;
    __syncthreads();
    part[t] += add;
    __syncthreads();
  }
  int acc = part[t] - sum;                                // exclusive
  for (int64_t i = lo; i < hi; ++i) {
    const int c = hist[i];
    hist[i] = acc;
    acc += c;
  }
  __threadfence_block();
  __syncthreads();
  for (int r = t; r < R; r += 1024) grp_off[r] = hist[(int64_t)r * nb];
  if (t == 0) grp_off[R] = (int)N;
}

// One wave per block, walking its candidates in order 64 at a time: lanes
// holding the same request take consecutive slots from that request's
// cursor in lane order (ballot ranks), so the order within a request is
// the original one.
__global__ __launch_bounds__(64) void group_scatter(const int32_t* __restrict__ ids, int64_t N,
                                                    int R, int64_t G, int nb,
                                                    const int32_t* __restrict__ base,
                                                    int32_t* __restrict__ order) {
  __shared__ int cursor[kGroupMaxRequests];
  const int b = blockIdx.x, lane = threadIdx.x;
  for (int r = lane; r < R; r += 64) cursor[r] = base[(int64_t)r * nb + b];
  __syncthreads();
  const int64_t lo = (int64_t)b * G, hi = min(lo + G, N);
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int64_t c = lo; c < hi; c += 64) {
    const int64_t i = c + lane;
    const bool valid = i < hi;
    const int key = valid ? clamp_request(ids[i], R) : -1;
    uint64_t todo = __ballot(valid);
    while (todo != 0) {
      const int leader = __builtin_ctzll(todo);
      const int k0 = __shfl(key, leader);
      const uint64_t same = __ballot(valid && key == k0);
      const int at = cursor[k0];                          // read by every lane first ...
      if (valid && key == k0) order[at + __builtin_popcountll(same & below)] = (int)i;
      if (lane == leader) cursor[k0] = at + __builtin_popcountll(same);   // ... then advanced
      todo &= ~same;
    }
  }
}

// ---------------------------------------------------------------------------
// Tile plan for one batch (one workgroup of 256 threads, one wave per SIMD):
// every request's history length and tile count are read in one pass; the
// requests are sorted by (history length descending, index) as 32-bit keys
// in LDS (kPlanLenBits bits of clamped length, 12 bits of index): up to 256
// requests by counting each key's rank, more with a bitonic sort; an
// exclusive scan of the tile counts in that order gives P. Beyond
// kAttnPlanMaxSort requests only the header is written (mode 0: the kernel
// keeps its built-in order).
// ---------------------------------------------------------------------------
constexpr int kPlanThreads = 256;
constexpr int kPlanIdBits = 12;
constexpr int kPlanLenBits = 32 - kPlanIdBits;   // lengths beyond 2^20 - 1 tie
static_assert(kAttnPlanMaxSort == (1 << kPlanIdBits), "plan key layout");

__global__ __launch_bounds__(kPlanThreads) void attn_plan_kernel(
    const int32_t* __restrict__ cand_off, const int32_t* __restrict__ kv_off, int R, int Tq,
    int H, int32_t* __restrict__ plan) {
  constexpr int PER = (int)kAttnPlanMaxSort / kPlanThreads;   // sorted positions per thread
  constexpr uint32_t kLenMax = (1u << kPlanLenBits) - 1;
  __shared__ __attribute__((aligned(16))) uint32_t key[kAttnPlanMaxSort];
  __shared__ int32_t tiles[kAttnPlanMaxSort];
  __shared__ int32_t wsum[kPlanThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (R > kAttnPlanMaxSort) {
    if (tid < kPlanHeader) plan[tid] = tid == 2 ? R : 0;   // mode 0
    return;
  }
  int32_t* ids = plan + kPlanHeader;
  int32_t* P = ids + R;
  if (R <= kPlanThreads) {
    // Up to one request per thread: its sorted position is the number of
    // smaller keys (keys are distinct), counted over the LDS copy four keys
    // per read; then the tile counts are scanned in sorted order.
    uint32_t kk = ~0u;
    int tl = 0;
    if (tid < R) {
      const uint32_t L = (uint32_t)max(kv_off[tid + 1] - kv_off[tid], 0);
      const int64_t rows = (int64_t)max(cand_off[tid + 1] - cand_off[tid], 0) * Tq;
      kk = ((kLenMax - min(L, kLenMax)) << kPlanIdBits) | (uint32_t)tid;
      tl = (int)((rows + kAttnTileRows - 1) / kAttnTileRows) * H;
    }
    key[tid] = kk;                                         // padding: ~0, never smaller
    __syncthreads();
    int rank = 0;
    const uint4* k4 = reinterpret_cast<const uint4*>(key);
#pragma unroll 8
    for (int c = 0; c < kPlanThreads / 4; ++c) {
      const uint4 q = k4[c];
      rank += (q.x < kk) + (q.y < kk) + (q.z < kk) + (q.w < kk);
    }
    if (tid < R) {
      tiles[rank] = tl;
      ids[rank] = tid;
    }
    __syncthreads();
    const int t = tid < R ? tiles[tid] : 0;
    int incl = t;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(incl, o);
      if (lane >= o) incl += y;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    int run = incl - t;
    for (int w = 0; w < wave; ++w) run += wsum[w];
    if (tid < R) P[tid] = run;
    if (tid == R - 1) {
      P[R] = run + t;
      plan[1] = run + t;
    }
    if (tid == 0) {
      if (R == 0) {
        P[0] = 0;
        plan[1] = 0;
      }
      plan[0] = 1;
      plan[2] = R;
      plan[3] = H;
      plan[4] = Tq;
      plan[5] = kAttnTileRows;
      plan[6] = 0;
      plan[7] = 0;
    }
    return;
  }
  int n = 1;
  while (n < R) n <<= 1;
  for (int i = tid; i < n; i += kPlanThreads) {
    uint32_t kk = ~0u;                                     // padding sorts last
    if (i < R) {
      const uint32_t L = (uint32_t)max(kv_off[i + 1] - kv_off[i], 0);
      const int64_t rows = (int64_t)max(cand_off[i + 1] - cand_off[i], 0) * Tq;
      kk = ((kLenMax - min(L, kLenMax)) << kPlanIdBits) | (uint32_t)i;
      tiles[i] = (int)((rows + kAttnTileRows - 1) / kAttnTileRows) * H;
    }
    key[i] = kk;
  }
  __syncthreads();
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = tid; i < n / 2; i += kPlanThreads) {
        const int lo = 2 * i - (i & (stride - 1)), hi = lo + stride;
        const uint32_t x = key[lo], y = key[hi];
        if ((x > y) == ((lo & size) == 0)) {
          key[lo] = y;
          key[hi] = x;
        }
      }
      __syncthreads();
    }
  }
  // Thread tid owns sorted positions PER tid .. PER tid + PER - 1.
  int cnt[PER], rid[PER], tsum = 0;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int i = PER * tid + e;
    rid[e] = i < R ? (int)(key[i] & ((1u << kPlanIdBits) - 1)) : 0;
    cnt[e] = i < R ? tiles[rid[e]] : 0;
    tsum += cnt[e];
  }
  // Block exclusive scan of the per-thread sums.
  int incl = tsum;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  int run = incl - tsum;
  for (int w = 0; w < wave; ++w) run += wsum[w];
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int i = PER * tid + e;
    if (i < R) {
      ids[i] = rid[e];
      P[i] = run;
    }
    run += cnt[e];
  }
  if (tid == kPlanThreads - 1) {
    P[R] = run;
    plan[0] = 1;
    plan[1] = run;
    plan[2] = R;
    plan[3] = H;
    plan[4] = Tq;
    plan[5] = kAttnTileRows;
    plan[6] = 0;
    plan[7] = 0;
  }
}

template <int D, bool MAPPED, bool QPROJ = false>
hipError_t launch_fast(const AttentionArgs& a, const int32_t* cand_off, const int32_t* order,
                       hipStream_t s) {
  constexpr int W = attn_waves<D>(), TR = 32 * W;
  const int64_t slots = a.R + (a.N * a.q_len + TR - 1) / TR;
  constexpr int64_t kRound = (int64_t)kNumXcd * kPlanChunk;
  const int32_t* plan = MAPPED ? nullptr : a.plan;
  const int64_t grid = plan != nullptr ? (slots * a.heads + kRound - 1) / kRound * kRound
                                       : slots * a.heads;
  const float scale_log2 = a.scale * 1.4426950408889634f;
  if (!grid_fits(grid, 64 * W)) return hipErrorInvalidConfiguration;
  return launch_kernel(dca_attn_bf16<D, W, MAPPED, QPROJ>, dim3((uint32_t)grid), dim3(64 * W), s,
                       static_cast<const bf16_t*>(a.q), static_cast<const bf16_t*>(a.k),
                       static_cast<const bf16_t*>(a.v), cand_off, a.kv_offsets,
                       static_cast<bf16_t*>(a.out), (int)a.R, a.q_len, a.heads, a.kv_stride,
                       scale_log2, slots, order, static_cast<const bf16_t*>(a.residual),
                       static_cast<bf16_t*>(a.out_sum), static_cast<const bf16_t*>(a.proj_w),
                       plan);
}

// The mapped form on the tiled kernel: group, then attend in grouped order.
template <int D>
hipError_t launch_fast_mapped(const AttentionArgs& a, hipStream_t s) {
  int64_t G = 0;
  int nb = 0;
  if (!mapped_grouping_plan(a.R, a.N, &G, &nb)) return hipErrorInvalidValue;
  char* ws = static_cast<char*>(a.workspace);
  int32_t* grp_off = reinterpret_cast<int32_t*>(ws);
  int32_t* order = reinterpret_cast<int32_t*>(ws + align_up256((size_t)(a.R + 1) * 4));
  int32_t* hist = reinterpret_cast<int32_t*>(ws + align_up256((size_t)(a.R + 1) * 4) +
                                             align_up256((size_t)a.N * 4));
  hipError_t e = launch_kernel(group_count, dim3((uint32_t)nb), dim3(256), s, a.ids, a.N,
                               (int)a.R, G, nb, hist);
  if (e == hipSuccess)
    e = launch_kernel(group_scan, dim3(1), dim3(1024), s, hist, a.R * (int64_t)nb, (int)a.R, nb,
                      a.N, grp_off);
  if (e == hipSuccess)
    e = launch_kernel(group_scatter, dim3((uint32_t)nb), dim3(64), s, a.ids, a.N, (int)a.R, G,
                      nb, static_cast<const int32_t*>(hist), order);
  if (e != hipSuccess) return e;
  return launch_fast<D, true>(a, grp_off, order, s);
}

template <typename T>
hipError_t launch_generic(const AttentionArgs& a, hipStream_t s) {
  if (!grid_fits(a.N * a.q_len, 64) || a.heads > 65535) return hipErrorInvalidConfiguration;
  return launch_kernel(dca_attn_generic<T>, dim3((uint32_t)(a.N * a.q_len), (uint32_t)a.heads),
                       dim3(64), s, static_cast<const T*>(a.q), static_cast<const T*>(a.k),
                       static_cast<const T*>(a.v), a.cand_offsets, a.kv_offsets,
                       static_cast<T*>(a.out), (int)a.R, a.q_len, a.heads, a.head_dim,
                       a.kv_stride, a.scale, a.ids, static_cast<const T*>(a.residual),
                       static_cast<T*>(a.out_sum), static_cast<const T*>(a.proj_w), a.proj_in);
}

}  // namespace

bool mapped_grouping_plan(int64_t R, int64_t N, int64_t* G, int* nb) {
  if (R < 1 || R > kGroupMaxRequests || N < 1) return false;
  int64_t g = 4096;
  while (R * ((N + g - 1) / g) > kGroupMaxHist && g < (int64_t(1) << 24)) g *= 2;
  const int64_t blocks = (N + g - 1) / g;
  if (R * blocks > kGroupMaxHist || blocks >= (int64_t(1) << 31)) return false;
  *G = g;
  *nb = (int)blocks;
  return true;
}

size_t mapped_grouping_bytes(int64_t R, int64_t N) {
  int64_t G = 0;
  int nb = 0;
  if (!mapped_grouping_plan(R, N, &G, &nb)) return 0;
  return align_up256((size_t)(R + 1) * 4) + align_up256((size_t)N * 4) +
         align_up256((size_t)R * (size_t)nb * 4);
}

size_t attention_plan_bytes(int64_t R) {
  return align_up256((size_t)(kPlanHeader + 2 * R + 1) * sizeof(int32_t));
}

hipError_t launch_attention_plan(const int32_t* cand_off, const int32_t* kv_off, int64_t R,
                                 int q_len, int heads, int32_t* plan, hipStream_t s) {
  return launch_kernel(attn_plan_kernel, dim3(1), dim3(kPlanThreads), s, cand_off, kv_off,
                       (int)R, q_len, heads, plan);
}

hipError_t launch_attention(const AttentionArgs& a, bool fast, hipStream_t s) {
  // The tiled kernel runs on request-contiguous candidates: the CSR offsets,
  // or a caller's per-candidate map grouped by request first (that needs the
  // grouping workspace); otherwise the general kernel runs.
  if (a.proj_w != nullptr) {
    // Fused query projection: the tiled kernel for head_dim 64 and a
    // projection input of kProjIn, the general kernel otherwise.
    if (fast && a.ids == nullptr && a.head_dim == 64 && a.proj_in == kProjIn)
      return launch_fast<64, false, true>(a, a.cand_offsets, nullptr, s);
    return a.bf16 ? launch_generic<bf16_t>(a, s) : launch_generic<float>(a, s);
  }
  if (fast && a.ids == nullptr)
    return a.head_dim == 128 ? launch_fast<128, false>(a, a.cand_offsets, nullptr, s)
                             : launch_fast<64, false>(a, a.cand_offsets, nullptr, s);
  if (fast && a.workspace != nullptr)
    return a.head_dim == 128 ? launch_fast_mapped<128>(a, s) : launch_fast_mapped<64>(a, s);
  return a.bf16 ? launch_generic<bf16_t>(a, s) : launch_generic<float>(a, s);
}

}  // namespace rocs
