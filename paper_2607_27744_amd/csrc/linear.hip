// IKBO fused linear (Eq. glm-linear, two-group case; Section 4.1 decomposition;
// broadcast-add fused into the GEMM epilogue, Section 4.2.1).
//
//   out[n][d] = act( sum_k W_CC[d][k] xc[n][k] + Z[m_n][d] + b[d] ),
//   Z = X^R W_CR^T computed once per request (batch size R).
//
// Two launches on the caller's stream:
//   1. request side: Z (fp32, [R, D]) on the matrix cores, plus the expanded
//      index map ids[n] = m_n, in one grid;
//   2. candidate side: a bf16 MFMA GEMM over the candidate batch whose
//      accumulators start from Z[m_n] + b, so the request term is added in
//      registers and only the final activations are written.
// The general (fp32 / unaligned) path keeps the same two-step structure with
// plain FMA kernels.
#include "common.h"
#include "kernels.h"
#include "launch.h"

#include <atomic>
#include <random>

namespace rocs {
namespace {

// ---------------------------------------------------------------------------
// Index map expansion (standalone; also used by rocs_request_ids).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void request_ids_kernel(const int32_t* __restrict__ off, int R,
                                                          int64_t N, int32_t* __restrict__ ids) {
  const int64_t n = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (n < N) ids[n] = owner_of(off, R, n);
}

// ---------------------------------------------------------------------------
// Request-side GEMM, bf16 in: the request table Zb = X^R W_CR^T + b (fp32;
// the bias is folded in here, once per request) and, for a full GLM layer,
// the request-side output Y^R = act(X^R W_RR^T + b^R) (bf16) from the same
// launch: the stacked weight [W_RR; W_CR] of Section 4.1, one GEMM at batch
// size R. One workgroup per 16 x 16 output tile (the W_RR column tiles come
// first); its four waves split K in 32-wide steps (operands straight from
// global memory into MFMA registers, each lane's 8 consecutive k are one
// 16-byte load) and reduce through LDS in a fixed order. Workgroups past the
// tiles expand the index map when the candidate GEMM needs it.
// ---------------------------------------------------------------------------
struct RequestOut {          // the optional Y^R part of the stacked weight
  const bf16_t* w;           // W_RR [d, K]
  const float* bias;         // b^R [d] or NULL
  bf16_t* y;                 // Y^R [R, d]
  int d, tiles, relu;        // tiles = ceil(d / 16); 0 when there is no Y^R
};

// One 16 x 16 output tile `tile` of the stacked request GEMM, by a 256-thread
// workgroup; `red` is 4 KiB of LDS. Returns whether the tile was a Zb tile
// (the candidate side's input) and, for wave 0, its (row block, column block).
__device__ __forceinline__ bool request_tile(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ w_in,
    const float* __restrict__ bias_in, float* __restrict__ z, int R, int K, int D_in,
    int tiles_d, const RequestOut& yr, int tile, ROCS_LDS f32x4* red) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int tiles_all = yr.tiles + tiles_d;
  const int t = tile % tiles_all;
  const bool to_y = t < yr.tiles;                 // a column tile of Y^R
  const bf16_t* w = to_y ? yr.w : w_in;
  const float* bias = to_y ? yr.bias : bias_in;
  const int D = to_y ? yr.d : D_in;
  const int r0 = (tile / tiles_all) * 16, d0 = (to_y ? t : t - yr.tiles) * 16;
  const int row = lane & 15, kq = (lane >> 4) * 8;
  const bool dok = d0 + row < D, rok = r0 + row < R;
  const bf16_t* wp = w + (int64_t)(d0 + row) * K + kq;
  const bf16_t* xp = x + (int64_t)(r0 + row) * K + kq;
  // Four waves split K; in a larger workgroup (the streaming kernel's) the
  // other waves only join the barriers, so both launch forms sum alike.
  if (wave < 4) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (int k = wave * 32; k < K; k += 128) {
      const bool kok = k + kq < K;
      const bf16x8 a = as_bf16x8(load16(wp + k, dok && kok));
      const bf16x8 b = as_bf16x8(load16(xp + k, rok && kok));
      acc = mfma16(a, b, acc);   // acc[i] = Z[r0 + row][d0 + 4 (lane / 16) + i]
    }
    red[wave * kWave + lane] = acc;
  }
  __syncthreads();
  if (wave == 0) {
    f32x4 s = ((red[lane] + red[kWave + lane]) + red[2 * kWave + lane]) + red[3 * kWave + lane];
    const int d = d0 + (lane >> 4) * 4;
    if (rok && d < D) {
      if (bias != nullptr) s += *reinterpret_cast<const f32x4*>(bias + d);
      if (to_y) {
        if (yr.relu) s = f32x4{fmaxf(s[0], 0.f), fmaxf(s[1], 0.f), fmaxf(s[2], 0.f), fmaxf(s[3], 0.f)};
        *reinterpret_cast<u32x2*>(yr.y + (int64_t)(r0 + row) * D + d) =
            u32x2{pack_bf16x2(s[0], s[1]), pack_bf16x2(s[2], s[3])};
      } else {
        *reinterpret_cast<f32x4*>(z + (int64_t)(r0 + row) * D + d) = s;
      }
    }
  }
  return !to_y;
}

__global__ __launch_bounds__(256) void request_gemm_bf16(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ w_in, const float* __restrict__ bias_in,
    float* __restrict__ z, const int32_t* __restrict__ off, int32_t* __restrict__ ids, int R,
    int64_t N, int K, int D_in, int tiles_d, int z_blocks, RequestOut yr) {
  if ((int)blockIdx.x >= z_blocks) {
    const int64_t n = (int64_t)(blockIdx.x - z_blocks) * 256 + threadIdx.x;
    if (n < N) ids[n] = owner_of(off, R, n);
    return;
  }
  __shared__ f32x4 red[4 * kWave];
  request_tile(x, w_in, bias_in, z, R, K, D_in, tiles_d, yr, (int)blockIdx.x, (ROCS_LDS f32x4*)red);
}

// ---------------------------------------------------------------------------
// Candidate-side GEMM with the fused request broadcast, bf16 MFMA 32x32x16.
//
// Matrix-core roles: A = W_CC rows (output features d), B = candidate rows,
// so each lane's accumulator holds, for one candidate, four runs of 4
// consecutive output features (8-byte bf16 stores). Workgroup tile BM
// (features) x BN (candidates), WAVES_M x WAVES_N waves, K staged through
// double-buffered LDS in BK-wide slabs; the next slab is prefetched into
// registers while the current one feeds the MFMAs. LDS rows carry a 16-byte
// pad so the rows read by one fragment load spread over all banks.
//
// Epilogue fusion: accumulators are initialised with Z[m_n][d] + b[d] before
// the K loop (so these loads overlap the first slab's loads), and the
// epilogue only applies the activation, rounds and stores. A tile whose rows
// all belong to one request (the common case: requests hold hundreds to tens
// of thousands of candidates) loads each Z row segment once for all its rows.
// ---------------------------------------------------------------------------
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, bool HAS_ADD>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N) __attribute__((amdgpu_waves_per_eu(2)))
void ikbo_gemm_bf16(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ xadd, const bf16_t* __restrict__ w,
    const float* __restrict__ bias, const float* __restrict__ z, const int32_t* __restrict__ ids,
    bf16_t* __restrict__ out, int64_t N, int K, int D, int tiles_m, int relu, int R,
    int ids_sorted) {
  constexpr int NT = 64 * WAVES_M * WAVES_N;
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int ROW = BK + 8;                 // LDS row (bf16) with 16-byte pad
  constexpr int CPR = BK / 8;                 // 16-byte chunks per slab row
  constexpr int RPP = NT / CPR;               // slab rows staged per pass
  constexpr int CA = BM / RPP, CB = BN / RPP;
  static_assert(BM % RPP == 0 && BN % RPP == 0, "staging does not tile");
  static_assert(WM % 32 == 0 && WN % 32 == 0 && BK % 16 == 0, "MFMA tiling");
  __shared__ __attribute__((aligned(16))) bf16_t lds_a[2][BM][ROW];
  __shared__ __attribute__((aligned(16))) bf16_t lds_b[2][BN][ROW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint32_t tile = xcd_remap(blockIdx.x, gridDim.x);
  const int m0 = (int)(tile % (uint32_t)tiles_m) * BM;
  const int64_t n0 = (int64_t)(tile / (uint32_t)tiles_m) * BN;
  const int wm0 = (wave % WAVES_M) * WM, wn0 = (wave / WAVES_M) * WN;
  const int l32 = lane & 31, h4 = (lane >> 5) * 4, h8 = (lane >> 5) * 8;

  const int srow = tid / CPR, skc = (tid % CPR) * 8;
  u32x4 ra[CA], rb[CB];
  auto load_slab = [&](int k0) {
    const bool kok = k0 + skc < K;
#pragma unroll
    for (int i = 0; i < CA; ++i) {
      const int d = m0 + srow + RPP * i;
      ra[i] = load16(w + (int64_t)d * K + k0 + skc, kok && d < D);
    }
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int64_t n = n0 + srow + RPP * i;
      const bool ok = kok && n < N;
      const int64_t o = n * K + k0 + skc;
      if constexpr (HAS_ADD) {
        // GLM pointwise residual: round(x + x_add) elementwise, in fp32.
        const u32x4 p = load16(x + o, ok), q = load16(xadd + o, ok);
        u32x4 s;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          s[e] = pack_bf16x2(bf16_lo(p[e]) + bf16_lo(q[e]), bf16_hi(p[e]) + bf16_hi(q[e]));
        rb[i] = s;
      } else {
        rb[i] = load16(x + o, ok);
      }
    }
  };
  auto store_slab = [&](int buf) {
#pragma unroll
    for (int i = 0; i < CA; ++i)
      *reinterpret_cast<u32x4*>(&lds_a[buf][srow + RPP * i][skc]) = ra[i];
#pragma unroll
    for (int i = 0; i < CB; ++i)
      *reinterpret_cast<u32x4*>(&lds_b[buf][srow + RPP * i][skc]) = rb[i];
  };

  const int nk = (K + BK - 1) / BK;
  load_slab(0);

  // Accumulators start at b[d] + Z[m_n][d]; element 4 q + i of tile (fm, fn)
  // is feature m0 + wm0 + 32 fm + 8 q + h4 + i of candidate n0 + wn0 + 32 fn + l32.
  f32x16 acc[FM][FN];
  {
    // A request id outside [0, R) (a malformed caller map) is clamped into
    // range: wrong rows, never an access outside Z.
    auto req = [&](int64_t n) { return (int)min((uint32_t)ids[n], (uint32_t)(R - 1)); };
    // Sorted ids (expanded from CSR offsets): equal first and last ids mean
    // the whole tile has one request. A caller's map has no such order.
    const bool one_request = z != nullptr && ids_sorted != 0 &&
                             ids[n0] == ids[(n0 + BN < N ? n0 + BN : N) - 1];
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int64_t n = n0 + wn0 + 32 * fn + l32;
      const float* zr = nullptr;
      if (z != nullptr) {
        const int r = one_request ? req(n0) : (n < N ? req(n) : 0);
        zr = z + (int64_t)r * D;
      }
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int d = m0 + wm0 + 32 * fm + 8 * q + h4;
          f32x4 v = {0.f, 0.f, 0.f, 0.f};
          if (d < D) {
            if (bias != nullptr) v = *reinterpret_cast<const f32x4*>(bias + d);
            if (zr != nullptr && (one_request || n < N)) v += *reinterpret_cast<const f32x4*>(zr + d);
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[fm][fn][4 * q + i] = v[i];
        }
    }
  }

  store_slab(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load_slab((kt + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 af[FM], bfr[FN];
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
        af[fm] = *reinterpret_cast<const bf16x8*>(&lds_a[cur][wm0 + 32 * fm + l32][ks * 16 + h8]);
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
        bfr[fn] = *reinterpret_cast<const bf16x8*>(&lds_b[cur][wn0 + 32 * fn + l32][ks * 16 + h8]);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = mfma32(af[fm], bfr[fn], acc[fm][fn]);
    }
    if (kt + 1 < nk) store_slab(cur ^ 1);
    __syncthreads();
  }

  // Epilogue: activation, round to bf16, 8-byte stores.
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    const int64_t n = n0 + wn0 + 32 * fn + l32;
    if (n >= N) continue;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int d = m0 + wm0 + 32 * fm + 8 * q + h4;
        if (d >= D) continue;
        float v[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = relu ? fmaxf(acc[fm][fn][4 * q + i], 0.f) : acc[fm][fn][4 * q + i];
        *reinterpret_cast<u32x2*>(out + n * D + d) =
            u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
      }
  }
}

// ---------------------------------------------------------------------------
// Streaming candidate GEMM (bf16, K a multiple of 64), the main path.
//
// Persistent workgroups, one per CU, walk the 256 (features) x 256
// (candidates) output tiles with a stride of the grid; eight waves, two per
// SIMD, each own a 64 x 128 block (8 MFMA 32x32 accumulators, 128 of the
// wave's 256 registers), so one wave's stalls (fragment reads, the
// epilogue's stores) leave the SIMD to the other. K arrives in 64-wide slabs
// (128-byte row segments: whole cache lines, which the L2 serves at twice the
// rate of half lines) through LDS rings filled by LDS DMA loads, as one
// stream across tile boundaries: the weight slab (L2-resident) one slab ahead
// of use in a 2-deep ring, the candidate slab (from HBM, longer latency) two
// slabs ahead in a 3-deep ring; together exactly the 160 KiB of LDS. The
// 16-byte chunks of each slab row are XOR-swizzled by (row / 2) % 8, which
// puts the 16 rows read by each quarter-wave on distinct banks; fragments
// are read one k-step ahead.
//
// Producer waves: waves 0-3 issue every DMA load (two pieces between
// consecutive MFMA groups), waves 4-7 none. The two waves of a SIMD do not
// progress alike (the arbiter favours the older one, waves 0-3), so loads
// issued by the slower waves arrived late and the whole workgroup waited at
// the slab barrier for them; the faster waves have that time to spare. Each
// wave waits only for its own loads (the vector-memory counter is per wave),
// so waves 4-7 never wait on a load of the ring.
// IKBO tiling (Section 4.2.1): with a request term, tiles never straddle two
// requests: request r owns tile slots r + floor(off[r] / 256) ... (the last
// one partial), so the whole tile shares one row of the request table
// Zb = X^R W_CR^T + b, added in the epilogue (the broadcast add fused into
// the GEMM). Without a request term the tiles cover the candidate rows
// contiguously and Zb is the bias (or absent).
//
// Epilogue: Zb, activation on packed bf16, then the two wave halves swap
// 8-byte pieces so every lane holds 8 consecutive features of one row. Stored
// from that layout, each instruction would write 32 bytes into each of 32
// rows, and a CU then stores at about a quarter of the rate it reaches with
// whole 128-byte lines (measured on this part: ~38 GB/s against ~150 GB/s
// per CU). So each wave passes its block through 4 KiB of the candidate slot
// the last slab has just released (after a barrier): 32 rows at a time
// written in that layout, read back row-contiguous, and stored as 8 rows x
// 128 bytes per instruction.
//
// Rows past the tile's end are clamped loads whose results are not stored.
// ---------------------------------------------------------------------------
constexpr int kStreamBM = 256, kStreamBN = 256, kStreamBK = 64;
constexpr int kCpolNT = 2;   // buffer-instruction cache policy bits: NT (the former SLC bit)

// ReLU of two packed bf16 values: as 16-bit integers the negative values
// (sign bit set) are exactly those below zero, so a packed integer max with
// zero clamps them (and -0) to +0. Written as the one instruction: the
// compiler's own lowering of a packed max on a bit-cast pair has been seen
// to drop the second word of the pair.
__device__ __forceinline__ uint32_t relu_bf16x2(uint32_t p) {
  uint32_t r;
  asm("v_pk_max_i16 %0, %1, 0" : "=v"(r) : "v"(p));
  return r;
}

struct StreamTile {
  int slot;       // tile slot (candidate block)
  int mb;         // feature block
  int r;          // request of the slot (0 without a request term)
  int64_t n0;     // first candidate row
  int rows;       // candidate rows in the tile
  int m0;         // first output feature
};

// Tiles are numbered slot * tiles_m + mb and a workgroup takes every
// grid-th one; the step is passed split into (slot, mb) parts so that no
// division runs on the device.
struct StreamStep {
  int slots, mbs;                  // grid = slots * tiles_m + mbs, mbs < tiles_m
};

__device__ __forceinline__ void stream_next(StreamTile& c, StreamStep st, int tiles_m) {
  c.slot += st.slots;
  c.mb += st.mbs;
  if (c.mb >= tiles_m) {
    c.mb -= tiles_m;
    ++c.slot;
  }
}

// Move `c` forward (in grid steps) to the first tile that holds candidate
// rows; false when the slots are exhausted. All values are wave-uniform.
template <typename OffPtr>
__device__ __forceinline__ bool stream_seek(StreamTile& c, StreamStep st, int n_slots,
                                            int tiles_m, OffPtr off, int R, int64_t N) {
  for (; c.slot < n_slots; stream_next(c, st, tiles_m)) {
    c.m0 = c.mb * kStreamBM;
    if (off != nullptr) {
      auto base_of = [&](int r) { return (int64_t)r + off[r] / kStreamBN; };   // tile slots
      while (c.r + 1 < R && base_of(c.r + 1) <= c.slot) ++c.r;
      const int64_t end = off[c.r + 1];
      c.n0 = (int64_t)off[c.r] + (c.slot - base_of(c.r)) * kStreamBN;
      if (c.n0 < end) {
        c.rows = (int)(end - c.n0 < kStreamBN ? end - c.n0 : kStreamBN);
        return true;
      }
    } else {
      c.n0 = (int64_t)c.slot * kStreamBN;
      c.rows = (int)(N - c.n0 < kStreamBN ? N - c.n0 : kStreamBN);
      return true;
    }
  }
  return false;
}

// The request side inside the candidate kernel (Section 4.2.3, combined
// request and candidate kernels): the stacked request GEMM's 16 x 16 tiles
// are computed first, by the workgroups taken in ascending order, and each
// Zb tile publishes a completion flag (agent-scope release: the tile's
// stores reach every XCD before the flag does). A workgroup then issues its
// first candidate loads and waits for the flags while they are in flight,
// then fences once (agent-scope acquire); the main loop and the epilogue
// carry no request-side state. Flags hold this call's epoch (a per-process
// random salt and a call counter), so stale flags from earlier calls never
// match and nothing resets them. The wait is bounded: past the limit the
// workgroup computes every tile whose flag is still unset itself (the same
// code, so the same values), so every workgroup always finishes.
struct FusedRequest {
  const bf16_t* x;           // x_req [R, K]
  const bf16_t* w;           // W_CR [D, K]
  const float* bias;         // b [D] or NULL
  float* z;                  // Zb [R, D] (workspace)
  RequestOut yr;             // optional Y^R part of the stacked weight
  uint64_t* flags;           // one per Zb tile: ceil(R / 16) x ceil(D / 16)
  uint64_t epoch;
  int K, tiles_d, n_tiles;   // n_tiles: all request tiles (Y^R and Zb)
};

constexpr int kFlagSpinLimit = 1 << 17;   // polls of about 0.3 us each

// This call's flag value: a per-process random salt in the high word and a
// call counter below it (never zero).
uint64_t next_epoch() {
  static std::atomic<uint64_t> counter{[] {
    std::random_device rd;
    return (uint64_t)rd() << 32 | 1u;
  }()};
  return counter.fetch_add(1, std::memory_order_relaxed);
}

template <bool HAS_ZB, bool RELU, bool FUSED>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void ikbo_gemm_stream(const bf16_t* __restrict__ x, const bf16_t* __restrict__ w,
                      const float* __restrict__ zb, const int32_t* __restrict__ off_g,
                      bf16_t* __restrict__ out, int R, int64_t N, int K, int D, int tiles_m,
                      int n_slots, StreamStep step_g, FusedRequest fr) {
  constexpr int BM = kStreamBM, BN = kStreamBN, BK = kStreamBK;
  constexpr int NSA = 2, NSB = 3;                // ring depths: weights, candidates
  constexpr int ROWB = BK * 2;                   // bytes of one slab row (128)
  constexpr int RPI = 1024 / ROWB;               // slab rows per wave-wide DMA load (8)
  constexpr int NI = BM / RPI / 8;               // DMA loads per wave and operand (4)
  constexpr int SLAB = BM * ROWB;                // bytes of one operand slab (32 KiB)
  constexpr int BBASE = NSA * SLAB;              // candidate ring after the weight ring
  static_assert(BM == BN && NI * RPI * 8 == BM && ROWB == 128, "tiling");
  static_assert((NSA + NSB) * SLAB <= 160 * 1024, "LDS");
  __shared__ __attribute__((aligned(1024))) char lds[(NSA + NSB) * SLAB];
  ROCS_LDS char* const lds3 = (ROCS_LDS char*)lds;
  // The offsets are read-only for the kernel's lifetime: read them through
  // the constant address space (scalar loads).
  const __attribute__((address_space(4))) int32_t* off =
      (const __attribute__((address_space(4))) int32_t*)off_g;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5, h4 = 4 * hh;
  const int wm0 = (wave & 3) * 64, wn0 = (wave >> 2) * 128;
  const int nk = K / BK;
  const int rowb = K * 2;
  const int logical = (int)xcd_remap(blockIdx.x, gridDim.x);
  // Request tiles reduce through the third candidate ring slot, which the
  // prologue leaves empty.
  ROCS_LDS f32x4* const red = (ROCS_LDS f32x4*)(lds3 + BBASE + 2 * SLAB);
  auto run_request_tile = [&](int t) __attribute__((always_inline)) {
    const bool is_zb = request_tile(fr.x, fr.w, fr.bias, fr.z, R, fr.K, D, fr.tiles_d, fr.yr,
                                    t, red);
    if (is_zb && threadIdx.x == 0) {      // wave 0 stored the tile
      const int tiles_all = fr.yr.tiles + fr.tiles_d;
      const int fi = (t / tiles_all) * fr.tiles_d + (t % tiles_all - fr.yr.tiles);
      __hip_atomic_store(fr.flags + fi, fr.epoch, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
  };
  if constexpr (FUSED) {
    for (int t = logical; t < fr.n_tiles; t += (int)gridDim.x) run_request_tile(t);
  }
  // Candidate tiles: descending for the workgroups that took request tiles
  // (they get the smaller share when the tiles do not divide evenly).
  const int first = FUSED ? (int)gridDim.x - 1 - logical : logical;
  const uint32_t lbase = lds_addr(lds);

  // DMA lane map (producer waves 0-3): load i of this wave fills slab rows
  // RPI (PI wave + i) + lane / 8, chunk position lane % 8, with chunk
  // (lane % 8) ^ ((row / 2) % 8). Rows past the operand's valid rows are
  // clamped to the last valid one.
  constexpr int PI = 2 * NI;                     // DMA loads per producer wave and operand (8)
  const bool producer = wave < 4;
  const int drow0 = RPI * PI * (wave & 3) + (lane >> 3);
  auto dma_piece = [&](const char* src, int rowlim, uint32_t dst, int i) __attribute__((always_inline)) {
    const int row = drow0 + RPI * i;
    const uint32_t chunk = 16u * (uint32_t)((lane & 7) ^ ((row >> 1) & 7));
    lds_dma16_sv(src, __umul24((uint32_t)min(row, rowlim), (uint32_t)rowb) + chunk,
                 dst + (uint32_t)(RPI * (PI * (wave & 3) + i) * ROWB));
  };
  auto dma_all = [&](const char* src, int rowlim, uint32_t dst) __attribute__((always_inline)) {
    if (producer) {
#pragma unroll
      for (int i = 0; i < PI; ++i) dma_piece(src, rowlim, dst, i);
    }
  };

  // The issue cursor walks the slab sequence two slabs ahead of compute and
  // plans the candidate slab; the weight slab of the same position follows
  // one slab later (weights sit in L2, candidates come from HBM).
  StreamTile ic{first / tiles_m, first % tiles_m, 0, 0, 0, 0};
  bool ic_live = stream_seek(ic, step_g, n_slots, tiles_m, off, R, N);
  int ic_s = 0;
  int buf_b = 0, buf_a = 0;              // ring slots of the next loads
  const char* a_next_src = nullptr;      // weight slab queued behind the candidates
  int a_next_lim = 0;
  bool a_queued = false;
  // Loads planned for the current slab: weights of slab g + 1, candidates
  // of slab g + 2. They are issued one at a time between the MFMAs.
  const char* pa_src = nullptr;
  int pa_lim = 0;
  uint32_t pa_dst = 0;
  bool pa_on = false;
  const char* pb_src = nullptr;
  int pb_lim = 0;
  uint32_t pb_dst = 0;
  bool pb_on = false;
  auto plan_b = [&]() __attribute__((always_inline)) {
    const int kb = ic_s * ROWB;
    pb_src = reinterpret_cast<const char*>(x + ic.n0 * K) + kb;
    pb_lim = ic.rows - 1;
    pb_dst = lbase + (uint32_t)(BBASE + buf_b * SLAB);
    pb_on = true;
    buf_b = buf_b == NSB - 1 ? 0 : buf_b + 1;
    a_next_src = reinterpret_cast<const char*>(w + (int64_t)ic.m0 * K) + kb;
    a_next_lim = D - 1 - ic.m0;
    a_queued = true;
    if (++ic_s == nk) {
      ic_s = 0;
      stream_next(ic, step_g, tiles_m);
      ic_live = stream_seek(ic, step_g, n_slots, tiles_m, off, R, N);
    }
  };
  auto plan_a = [&]() __attribute__((always_inline)) {
    pa_src = a_next_src;
    pa_lim = a_next_lim;
    pa_dst = lbase + (uint32_t)(buf_a * SLAB);
    pa_on = true;
    buf_a ^= 1;
    a_queued = false;
  };
  // Group p (0..7) of the planned loads, two pieces each: weights for
  // p < 4, candidates after.
  auto dma_plan_piece = [&](int p) __attribute__((always_inline)) {
    if (!producer) return;
    if (p < NI) {
      if (pa_on) {
        dma_piece(pa_src, pa_lim, pa_dst, 2 * p);
        dma_piece(pa_src, pa_lim, pa_dst, 2 * p + 1);
      }
    } else {
      if (pb_on) {
        dma_piece(pb_src, pb_lim, pb_dst, 2 * (p - NI));
        dma_piece(pb_src, pb_lim, pb_dst, 2 * (p - NI) + 1);
      }
    }
  };

  // Fragment addresses within an operand slab: row 32 f + l32 of the wave's
  // quarter, chunk 2 ks + hh; the swizzle turns the ks step into XOR 32 ks.
  const uint32_t fa0 = (uint32_t)(l32 * ROWB + 16 * (hh ^ ((l32 >> 1) & 7)));
  f32x16 acc[2][4];
  int cbuf_a = 0, cbuf_b = 0;            // ring slots of the slab being computed
  // Fragments, double-buffered across k-steps (slot ks % 2): the reads of
  // step ks + 1 are in flight while the MFMAs of step ks run. The last
  // k-step of a slab that is not a tile's last is deferred: its fragments
  // are read (and waited for) before the slab barrier, and its MFMAs run
  // after the barrier, while the next slab's first fragment reads are in
  // flight; every wave would otherwise start each slab waiting for LDS. The
  // accumulation order is unchanged.
  bf16x8 af[2][2], bfr[2][4];
  auto compute = [&](auto first_slab, auto last_slab) __attribute__((always_inline)) {
    constexpr bool kFirst = decltype(first_slab)::value;
    constexpr bool kLastS = decltype(last_slab)::value;
    constexpr int KSTEPS = BK / 16;
    const uint32_t sa = (uint32_t)(cbuf_a * SLAB) + wm0 * ROWB;
    const uint32_t sb = (uint32_t)(BBASE + cbuf_b * SLAB) + wn0 * ROWB;
    auto load_frags = [&](int ks, int slot) __attribute__((always_inline)) {
#pragma unroll
      for (int f = 0; f < 4; ++f) {
        if (f < 2) af[slot][f] = *reinterpret_cast<const ROCS_LDS bf16x8*>(lds3 + sa + 32 * f * ROWB + (fa0 ^ (32u * ks)));
        bfr[slot][f] = *reinterpret_cast<const ROCS_LDS bf16x8*>(lds3 + sb + 32 * f * ROWB + (fa0 ^ (32u * ks)));
      }
    };
    // DMA group g (0..7) goes with the g-th MFMA group of the slab.
    constexpr int kDeferred = kFirst ? 0 : 2;          // MFMA groups of the previous slab
    load_frags(0, 0);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (!kFirst) {
#pragma unroll
      for (int fm = 0; fm < 2; ++fm) {
#pragma unroll
        for (int fn = 0; fn < 4; ++fn) acc[fm][fn] = mfma32(af[1][fm], bfr[1][fn], acc[fm][fn]);
        dma_plan_piece(fm);
        __builtin_amdgcn_sched_barrier(0x0002 | 0x0004);
      }
    }
    constexpr int KRUN = kLastS ? KSTEPS : KSTEPS - 1;
#pragma unroll
    for (int ks = 0; ks < KRUN; ++ks) {
      const int cur = ks & 1;
      if (ks + 1 < KSTEPS) load_frags(ks + 1, cur ^ 1);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int fm = 0; fm < 2; ++fm) {
#pragma unroll
        for (int fn = 0; fn < 4; ++fn) {
          if constexpr (kFirst) {
            if (ks == 0) {
              const f32x16 zero = {};
              acc[fm][fn] = mfma32(af[cur][fm], bfr[cur][fn], zero);
              continue;
            }
          }
          acc[fm][fn] = mfma32(af[cur][fm], bfr[cur][fn], acc[fm][fn]);
        }
        if (kDeferred + 2 * ks + fm < 8) dma_plan_piece(kDeferred + 2 * ks + fm);
        // Keep MFMAs and loads in this order; ALU work may move.
        __builtin_amdgcn_sched_barrier(0x0002 | 0x0004);
      }
    }
#pragma unroll
    for (int g = kDeferred + 2 * KRUN; g < 8; ++g) dma_plan_piece(g);
    // The deferred step's fragments are in registers before the barrier
    // hands this slab's ring slots to the next loads.
    if constexpr (!kLastS) wait_lgkmcnt0();
  };

  // Request row Zb[m0 + wm0 + 32 fm + 8 q + h4 .. +3] of the tile, loaded
  // after the tile's last MFMAs (the fragment registers are free then) and
  // added in the epilogue. The buffer's extent is the request's row, so
  // features past D read as zero.
  f32x4 zv[2][4];
  auto load_zb = [&](const StreamTile& c) __attribute__((always_inline)) {
    if constexpr (HAS_ZB) {
      const auto rz = buffer_rsrc(zb + (int64_t)c.r * D, (uint32_t)D * 4u);
      const uint32_t vo = 4u * (uint32_t)(c.m0 + wm0 + h4);
#pragma unroll
      for (int fm = 0; fm < 2; ++fm)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          zv[fm][q] = __builtin_bit_cast(
              f32x4, __builtin_amdgcn_raw_buffer_load_b128(rz, vo + 4u * (32 * fm + 8 * q), 0, 0));
    }
  };

  // Combined kernel: wait (bounded) until every Zb tile's flag carries this
  // call's epoch; past the limit, compute the missing tiles here.
  auto wait_request_side = [&]() __attribute__((always_inline)) {
    const int nflags = ((R + 15) / 16) * fr.tiles_d;
    int spins = 0;
    for (; spins < kFlagSpinLimit; ++spins) {
      bool ok = true;
      for (int i = lane; i < nflags; i += kWave)
        ok &= __hip_atomic_load(fr.flags + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == fr.epoch;
      if (__ballot(!ok) == 0) break;
      __builtin_amdgcn_s_sleep(8);
    }
    // Workgroup-wide verdicts go through one LDS word past the reduction
    // area, so every wave takes the same branch around the tiles' barriers.
    ROCS_LDS int* const verdict = (ROCS_LDS int*)(lds3 + BBASE + 2 * SLAB + 4096);
    if (threadIdx.x == 0) *verdict = 0;
    __syncthreads();
    if (lane == 0 && spins == kFlagSpinLimit) *verdict = 1;
    __syncthreads();
    const bool timed_out = *verdict != 0;
    __syncthreads();
    if (timed_out) {
      const int tiles_all = fr.yr.tiles + fr.tiles_d;
      for (int fi = 0; fi < nflags; ++fi) {
        if (threadIdx.x == 0)
          *verdict = __hip_atomic_load(fr.flags + fi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != fr.epoch;
        __syncthreads();
        const bool run = *verdict != 0;
        __syncthreads();
        if (run) run_request_tile((fi / fr.tiles_d) * tiles_all + fr.yr.tiles + fi % fr.tiles_d);
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  };

  // Epilogue. Element 4 q + i of acc[fm][fn] is feature 32 fm + 8 q + h4 + i
  // of candidate 32 fn + l32 (within the wave's block). For q = 2j, 2j + 1
  // the lower half-wave keeps its q = 2j words and takes the upper half's,
  // the upper half keeps q = 2j + 1 and takes the lower half's: then lane
  // (l32, hh) holds features 32 fm + 16 j + 8 hh .. +7, one 16-byte store.
  auto packed = [&](int fm, int fn, int q, uint32_t& lo, uint32_t& hi) __attribute__((always_inline)) {
    const f32x16& a = acc[fm][fn];
    float v0 = a[4 * q], v1 = a[4 * q + 1], v2 = a[4 * q + 2], v3 = a[4 * q + 3];
    if constexpr (HAS_ZB) {
      v0 += zv[fm][q][0];
      v1 += zv[fm][q][1];
      v2 += zv[fm][q][2];
      v3 += zv[fm][q][3];
    }
    lo = pack_bf16x2(v0, v1);
    hi = pack_bf16x2(v2, v3);
    if constexpr (RELU) {
      lo = relu_bf16x2(lo);
      hi = relu_bf16x2(hi);
    }
  };
  auto swapped = [&](int fm, int fn, int j) __attribute__((always_inline)) {
    uint32_t e0, e1, o0, o1;                     // words of q = 2j and q = 2j + 1
    packed(fm, fn, 2 * j, e0, e1);
    packed(fm, fn, 2 * j + 1, o0, o1);
    const auto s0 = __builtin_amdgcn_permlane32_swap(e0, o0, false, false);
    const auto s1 = __builtin_amdgcn_permlane32_swap(e1, o1, false, false);
    // Lower half: {own q = 2j, partner's q = 2j}; upper: {partner's q = 2j + 1, own}.
    const uint32_t w0 = s0[0], w2 = s0[1], w1 = s1[0], w3 = s1[1];
    return u32x4{w0, w1, w2, w3};
  };
  // A tile inside the row range of the output stores through a buffer
  // whose extent ends after the tile's last candidate row, so stores of rows
  // past it are dropped. A tile that reaches past feature D (D not a
  // multiple of the tile) tests each store.
  // `stage` is this wave's 4 KiB of free LDS. Staging layout: row r (of the
  // 32 candidates of one fn block) at r * 128 bytes, its 16-byte chunk c
  // (features 8 c .. 8 c + 7 of the wave's 64) at position c ^ (r % 8), so
  // both the writes (32 rows at one chunk) and the row-contiguous reads
  // (8 rows x 8 chunks) spread over all banks.
  auto store_tile = [&](const StreamTile& c, uint32_t stage) __attribute__((always_inline)) {
    if (c.m0 + BM <= D) {
      const auto ro = buffer_rsrc(out + c.n0 * D, (uint32_t)c.rows * (uint32_t)D * 2u);
      ROCS_LDS char* const st = lds3 + stage;
      const int rr = lane >> 3, cr = lane & 7;  // read-back: row 8 i + rr, chunk cr
      const uint32_t vo = 2u * ((uint32_t)(wn0 + rr) * (uint32_t)D + (uint32_t)(c.m0 + wm0 + 8 * cr));
#pragma unroll
      for (int fn = 0; fn < 4; ++fn) {
#pragma unroll
        for (int fm = 0; fm < 2; ++fm)
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const int ch = 4 * fm + 2 * j + hh;
            *reinterpret_cast<ROCS_LDS u32x4*>(st + l32 * 128 + 16 * (ch ^ (l32 & 7))) =
                swapped(fm, fn, j);
          }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = 8 * i + rr;
          const u32x4 v = *reinterpret_cast<const ROCS_LDS u32x4*>(st + r * 128 + 16 * (cr ^ (r & 7)));
          // Non-temporal (cache policy NT): the output is not read again by
          // this kernel, so it should not push the candidate slabs and the
          // weights out of L2 before the tile's other feature tiles read them.
          __builtin_amdgcn_raw_buffer_store_b128(
              v, ro, vo + 2u * (uint32_t)(32 * fn + 8 * i) * (uint32_t)D, 0, kCpolNT);
        }
      }
      return;
    }
#pragma unroll
    for (int fn = 0; fn < 4; ++fn) {
      const int rr = wn0 + 32 * fn + l32;
#pragma unroll
      for (int fm = 0; fm < 2; ++fm)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          // The swap is wave-wide: every lane takes part, only valid ones
          // store. D is a multiple of 4: a lane's 8 features are all valid,
          // or only the first 4 (the row's last ones).
          const u32x4 v = swapped(fm, fn, j);
          const int d = c.m0 + wm0 + 32 * fm + 16 * j + 8 * hh;
          if (rr < c.rows && d < D) {
            bf16_t* p = out + (c.n0 + rr) * D + d;
            if (d + 8 <= D) *reinterpret_cast<u32x4*>(p) = v;
            else *reinterpret_cast<u32x2*>(p) = u32x2{v[0], v[1]};
          }
        }
    }
  };

  // Prologue: candidates of slabs 0 and 1, weights of slab 0, all resident.
  if (!ic_live) return;
  StreamTile cc = ic;
  plan_b();
  plan_a();
  dma_all(pb_src, pb_lim, pb_dst);
  dma_all(pa_src, pa_lim, pa_dst);
  if (ic_live) {
    plan_b();
    dma_all(pb_src, pb_lim, pb_dst);
  }
  pa_on = pb_on = false;
  if constexpr (FUSED) wait_request_side();   // while the first slabs load
  wait_vmcnt<0>();
  ring_barrier();

  // One slab. Vector-memory operations retire in issue order (the
  // counter of outstanding ones is decremented in order), and only the
  // producer waves have ring loads in flight. In an inner slab the candidate
  // loads (slab g + 2) follow the weight loads (g + 1), so waiting until only
  // those are in flight makes slab g + 1 resident. In the last slab of a
  // tile the candidates of slab g + 2 wait until after the epilogue, and the
  // Zb loads are issued and drained with the slab; the epilogue stages
  // through the candidate slot the slab has just released, once every wave
  // is done with it.
  auto step = [&](auto first_slab, auto last_slab) __attribute__((always_inline)) {
    constexpr bool kLast = decltype(last_slab)::value;
    const bool a_next = a_queued;
    if (a_next) plan_a();
    const bool b_next = ic_live;
    if (!kLast && b_next) plan_b();
    compute(first_slab, last_slab);
    pa_on = pb_on = false;
    const uint32_t released = (uint32_t)(BBASE + cbuf_b * SLAB);
    cbuf_a ^= 1;
    cbuf_b = cbuf_b == NSB - 1 ? 0 : cbuf_b + 1;
    if constexpr (kLast) {
      ring_barrier();                            // every wave is past the slab's fragments
      load_zb(cc);
      wait_vmcnt<0>();
      store_tile(cc, released + (uint32_t)wave * 4096u);
      if (b_next) {
        plan_b();
        dma_all(pb_src, pb_lim, pb_dst);
        pb_on = false;
      }
    } else {
      if (producer) {
        if (b_next) wait_vmcnt<PI>(); else wait_vmcnt<0>();
      }
    }
    if (a_next) ring_barrier();                  // a next slab exists
  };
  while (true) {
    if (nk == 1) {
      step(std::true_type(), std::true_type());
    } else {
      step(std::true_type(), std::false_type());
      for (int s = 1; s < nk - 1; ++s) step(std::false_type(), std::false_type());
      step(std::false_type(), std::true_type());
    }
    stream_next(cc, step_g, tiles_m);
    if (!stream_seek(cc, step_g, n_slots, tiles_m, off, R, N)) break;
  }
}

// ---------------------------------------------------------------------------
// General path: any dtype, any K / D, no alignment requirements.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void request_gemm_generic(
    const T* __restrict__ x, const T* __restrict__ w, float* __restrict__ z,
    const int32_t* __restrict__ off, int32_t* __restrict__ ids, int R, int64_t N, int K, int D,
    int z_blocks) {
  if ((int)blockIdx.x >= z_blocks) {
    const int64_t n = (int64_t)(blockIdx.x - z_blocks) * 256 + threadIdx.x;
    if (n < N) ids[n] = owner_of(off, R, n);
    return;
  }
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)R * D) return;
  const int r = (int)(idx / D), d = (int)(idx % D);
  float acc = 0.f;
  for (int k = 0; k < K; ++k)
    acc = fmaf(load_f32(x + (int64_t)r * K + k), load_f32(w + (int64_t)d * K + k), acc);
  z[idx] = acc;
}

template <typename T>
__global__ __launch_bounds__(256) void linear_generic(
    const T* __restrict__ x, const T* __restrict__ xadd, const T* __restrict__ w,
    const float* __restrict__ bias, const float* __restrict__ z, const int32_t* __restrict__ ids,
    T* __restrict__ out, int64_t N, int K, int D, int relu, int R) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= N * D) return;
  const int64_t n = idx / D;
  const int d = (int)(idx % D);
  float acc = 0.f;
  for (int k = 0; k < K; ++k) {
    float xv = load_f32(x + n * K + k);
    if (xadd != nullptr) xv = (float)from_f32<T>(xv + load_f32(xadd + n * K + k));
    acc = fmaf(xv, load_f32(w + (int64_t)d * K + k), acc);
  }
  if (z != nullptr) acc += z[(int64_t)min((uint32_t)ids[n], (uint32_t)(R - 1)) * D + d];
  if (bias != nullptr) acc += bias[d];
  if (relu) acc = fmaxf(acc, 0.f);
  out[idx] = from_f32<T>(acc);
}

template <int BM, int BN, int BK, int WMW, int WNW>
hipError_t launch_fast_gemm(const LinearArgs& a, hipStream_t s) {
  const int tiles_m = (int)((a.d_out + BM - 1) / BM);
  const int64_t tiles_n = (a.N + BN - 1) / BN;
  const int64_t grid = tiles_m * tiles_n;
  if (!grid_fits(grid, 64 * WMW * WNW)) return hipErrorInvalidConfiguration;
  const bf16_t* x = static_cast<const bf16_t*>(a.x_cand);
  const bf16_t* xa = static_cast<const bf16_t*>(a.x_cand_add);
  const bf16_t* w = static_cast<const bf16_t*>(a.w_cand);
  bf16_t* o = static_cast<bf16_t*>(a.out);
  const float* z = a.k_req > 0 ? a.z : nullptr;
  if (xa != nullptr)
    return launch_kernel(ikbo_gemm_bf16<BM, BN, BK, WMW, WNW, true>, dim3((uint32_t)grid),
                         dim3(64 * WMW * WNW), s,
                         x, xa, w, a.bias, z, a.ids, o, a.N, (int)a.k_cand, (int)a.d_out,
                         tiles_m, (int)a.relu, (int)a.R, (int)!a.ids_given);
  return launch_kernel(ikbo_gemm_bf16<BM, BN, BK, WMW, WNW, false>, dim3((uint32_t)grid),
                       dim3(64 * WMW * WNW), s,
                       x, xa, w, a.bias, z, a.ids, o, a.N, (int)a.k_cand, (int)a.d_out,
                       tiles_m, (int)a.relu, (int)a.R, (int)!a.ids_given);
}

template <typename T>
hipError_t launch_generic(const LinearArgs& a, hipStream_t s) {
  hipError_t e = hipSuccess;
  if (a.k_req > 0) {
    if (!grid_fits((a.R * a.d_out + 255) / 256 + (a.N + 255) / 256, 256))
      return hipErrorInvalidConfiguration;
    const int z_blocks = (int)((a.R * a.d_out + 255) / 256);
    const int id_blocks = a.ids_given ? 0 : (int)((a.N + 255) / 256);
    e = launch_kernel(request_gemm_generic<T>, dim3(z_blocks + id_blocks), dim3(256), s,
                      static_cast<const T*>(a.x_req), static_cast<const T*>(a.w_req), a.z,
                      a.cand_offsets, a.ids, (int)a.R, a.N, (int)a.k_req, (int)a.d_out,
                      z_blocks);
    if (e != hipSuccess) return e;
  }
  const int64_t blocks = (a.N * a.d_out + 255) / 256;
  if (!grid_fits(blocks, 256)) return hipErrorInvalidConfiguration;
  return launch_kernel(linear_generic<T>, dim3((uint32_t)blocks), dim3(256), s,
                       static_cast<const T*>(a.x_cand), static_cast<const T*>(a.x_cand_add),
                       static_cast<const T*>(a.w_cand), a.bias,
                       a.k_req > 0 ? a.z : nullptr, a.ids, static_cast<T*>(a.out), a.N,
                       (int)a.k_cand, (int)a.d_out, (int)a.relu, (int)a.R);
}

}  // namespace

hipError_t launch_request_ids(const int32_t* off, int64_t R, int64_t N, int32_t* ids,
                              hipStream_t s) {
  if (!grid_fits((N + 255) / 256, 256)) return hipErrorInvalidConfiguration;
  return launch_kernel(request_ids_kernel, dim3((uint32_t)((N + 255) / 256)), dim3(256), s,
                       off, (int)R, N, ids);
}

hipError_t launch_request_table(const LinearArgs& a, hipStream_t s) {
  const int tiles_d = (int)((a.d_out + 15) / 16);
  if (!grid_fits((int64_t)tiles_d * ((a.R + 15) / 16), 256)) return hipErrorInvalidConfiguration;
  const int req_tiles = tiles_d * (int)((a.R + 15) / 16);
  const RequestOut none{nullptr, nullptr, nullptr, 0, 0, 0};
  return launch_kernel(request_gemm_bf16, dim3(req_tiles), dim3(256), s,
                       static_cast<const bf16_t*>(a.x_req), static_cast<const bf16_t*>(a.w_req),
                       a.bias, a.z, a.cand_offsets, a.ids, (int)a.R, a.N, (int)a.k_req,
                       (int)a.d_out, tiles_d, req_tiles, none);
}

hipError_t launch_linear(const LinearArgs& a, bool fast, hipStream_t s) {
  if (!fast) {
    if (a.y_req != nullptr) {
      // Y^R on the general path: the plain linear over the R request rows.
      LinearArgs r{};
      r.x_cand = a.x_req; r.w_cand = a.w_rr; r.bias = a.b_rr;
      r.N = a.R; r.k_cand = a.k_req; r.d_out = a.d_req; r.R = 1;
      r.bf16 = a.bf16; r.relu = a.relu; r.out = a.y_req;
      const hipError_t e = a.bf16 ? launch_generic<bf16_t>(r, s) : launch_generic<float>(r, s);
      if (e != hipSuccess || a.N == 0) return e;
    }
    return a.bf16 ? launch_generic<bf16_t>(a, s) : launch_generic<float>(a, s);
  }
  // The streaming kernel needs request-aligned tiles, i.e. CSR offsets; a
  // caller's per-candidate map takes the kernel with per-row request lookup.
  // (K and D bounds: the kernel's per-lane load and store offsets within a
  // 256-row tile are 32-bit.)
  const bool stream = !a.ids_given && a.x_cand_add == nullptr && a.k_cand % kStreamBK == 0 &&
                      a.k_cand < (int64_t(1) << 22) && a.d_out < (int64_t(1) << 22) &&
                      ((a.k_req > 0 ? a.R : 0) + (a.N + kStreamBN - 1) / kStreamBN) *
                              ((a.d_out + kStreamBM - 1) / kStreamBM) < (int64_t(1) << 31);
  // On request, the streaming kernel also runs the request side (combined
  // kernel); otherwise the request GEMM is a launch of its own. Separate
  // launches are the default on this part: the cross-XCD release / acquire
  // the combined kernel needs (an L2 write-back per request tile, an L2
  // invalidate per workgroup) costs more than the launch it saves.
  const bool fused = a.combined && stream && a.k_req > 0 && a.N > 0;
  RequestOut yr{static_cast<const bf16_t*>(a.w_rr), a.b_rr, static_cast<bf16_t*>(a.y_req),
                (int)a.d_req, a.y_req != nullptr ? (int)((a.d_req + 15) / 16) : 0, (int)a.relu};
  // No candidates: only the Y^R tiles (the request table has no reader).
  const int tiles_d = a.N > 0 ? (int)((a.d_out + 15) / 16) : 0;
  if (a.k_req > 0 && !grid_fits((int64_t)(yr.tiles + tiles_d) * ((a.R + 15) / 16) +
                                    (a.N + 255) / 256, 256))
    return hipErrorInvalidConfiguration;
  const int req_tiles = (yr.tiles + tiles_d) * (int)((a.R + 15) / 16);
  if (a.k_req > 0 && !fused) {
    const int id_blocks = stream || a.ids_given ? 0 : (int)((a.N + 255) / 256);
    hipError_t e = launch_kernel(request_gemm_bf16, dim3(req_tiles + id_blocks), dim3(256), s,
                                 static_cast<const bf16_t*>(a.x_req),
                                 static_cast<const bf16_t*>(a.w_req), a.bias, a.z,
                                 a.cand_offsets, a.ids, (int)a.R, a.N, (int)a.k_req,
                                 (int)a.d_out, tiles_d, req_tiles, yr);
    if (e != hipSuccess) return e;
  }
  if (a.N == 0) return hipSuccess;      // request-side output only
  if (stream) {
    const int tiles_m = (int)((a.d_out + kStreamBM - 1) / kStreamBM);
    const int64_t slots = (a.k_req > 0 ? a.R : 0) + (a.N + kStreamBN - 1) / kStreamBN;
    const int64_t n_tiles = slots * tiles_m;
    int cus = 0;
    const hipError_t e = current_cu_count(&cus);
    if (e != hipSuccess) return e;
    const int grid = (int)(n_tiles < cus ? n_tiles : cus);
    const StreamStep step{grid / tiles_m, grid % tiles_m};
    const float* zb = a.k_req > 0 ? a.z : a.bias;
    const int32_t* off = a.k_req > 0 ? a.cand_offsets : nullptr;
    const bf16_t* x = static_cast<const bf16_t*>(a.x_cand);
    const bf16_t* w = static_cast<const bf16_t*>(a.w_cand);
    bf16_t* o = static_cast<bf16_t*>(a.out);
    FusedRequest fr{};
    if (fused) {
      fr.x = static_cast<const bf16_t*>(a.x_req);
      fr.w = static_cast<const bf16_t*>(a.w_req);
      fr.bias = a.bias;
      fr.z = a.z;
      fr.yr = yr;
      fr.flags = reinterpret_cast<uint64_t*>(a.ids);   // the index map's slot is free here
      fr.epoch = next_epoch();
      fr.K = (int)a.k_req;
      fr.tiles_d = tiles_d;
      fr.n_tiles = req_tiles;
    }
    auto go = [&](auto kernel) {
      return launch_kernel(kernel, dim3((uint32_t)grid), dim3(512), s, x, w, zb, off, o,
                           (int)a.R, a.N, (int)a.k_cand, (int)a.d_out, tiles_m, (int)slots, step,
                           fr);
    };
    if (fused)
      return a.relu ? go(ikbo_gemm_stream<true, true, true>) : go(ikbo_gemm_stream<true, false, true>);
    if (zb != nullptr)
      return a.relu ? go(ikbo_gemm_stream<true, true, false>) : go(ikbo_gemm_stream<true, false, false>);
    return a.relu ? go(ikbo_gemm_stream<false, true, false>) : go(ikbo_gemm_stream<false, false, false>);
  }
  // Large tiles when they still give every CU at least four tiles. The bias
  // is already inside Z when there is a request term.
  LinearArgs b = a;
  if (a.k_req > 0) b.bias = nullptr;
  const int64_t big_tiles = ((a.d_out + 255) / 256) * ((a.N + 127) / 128);
  if (big_tiles >= 1024) return launch_fast_gemm<256, 128, 32, 2, 2>(b, s);
  return launch_fast_gemm<128, 128, 32, 2, 2>(b, s);
}

}  // namespace rocs
