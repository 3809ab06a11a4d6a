// IKBO linear compression block (LCB), two groups (Eq. glm-lcb,
// Eq. glm-lcb-two-groups; Section 4.1 decomposition, Section 4.2 IKBO).
//
//   Y^R_r = W_RR X^R_r                         once per request
//   Y^C_n = W_CR X^R_{m_n} + W_CC X^C_n          per candidate
//
// X^R_r [F_r, E] and X^C_n [F_c, E] are field x embedding matrices; the
// weights mix the field (row) axis. IKBO form: the request-side products
// Y^R and Z_r = W_CR X^R_r come out of one launch at batch size R (the
// stacked weight [W_RR; W_CR]); the candidate kernel computes W_CC X^C_n and
// adds Z_{m_n}, so no candidate-batched copy of X^R or Z exists.
#include "common.h"
#include "kernels.h"
#include "launch.h"

#include <type_traits>

namespace rocs {
namespace {

constexpr int kLcbWaves = 4;     // waves per workgroup; each streams its own candidates
constexpr int kLcbStages = 2;    // per-wave LDS ring depth (candidate inputs)

// ---------------------------------------------------------------------------
// Candidate kernel, bf16 MFMA (32x32x16): F_c = NK (multiple of 16), E in
// {64, 128}, O_c = 32 NOB.
//
// Per candidate the wave computes (Y^C_n)^T = (X^C_n)^T (W_CC)^T + Z^T:
//   A = (X^C_n)^T, rows = embedding columns, read with the transposing LDS
//       read out of the row-major [F_c, E] stage (no transpose in memory);
//   B = (W_CC)^T, held in registers for the whole run (the same key order
//       inside each 16-field step as the transposing read produces);
//   C starts at Z_{m_n}, kept in registers while the request stays the same.
// Each lane ends with runs of 4 consecutive embedding columns of one output
// field (16-byte Z loads). The output goes back through LDS: a half-wave
// swap gives each lane 16 contiguous bytes, written into the candidate's
// consumed input stage (XOR-swizzled by output row, conflict-free) and read
// back row-contiguous, so each store instruction writes 1 KiB of the
// candidate's contiguous output. Written straight from the MFMA layout, a
// store instruction would touch 32 rows with 16 bytes each, and the write
// path, not the matrix cores, would set the pace.
//
// Each wave owns a contiguous run of candidates and streams their inputs
// through a private 2-deep LDS ring with the DMA form of the global load
// (16 bytes per lane, chunks XOR-swizzled by field row), so no workgroup
// barrier is needed. The request of the next candidate follows by a forward
// walk over the CSR offsets (or the caller's per-candidate map).
// ---------------------------------------------------------------------------
template <int NK, int E, int NOB>
__global__ __launch_bounds__(64 * kLcbWaves) __attribute__((amdgpu_waves_per_eu(2)))
void lcb_cand_bf16(const bf16_t* __restrict__ xc, const bf16_t* __restrict__ wcc,
                   const float* __restrict__ z, const int32_t* __restrict__ off,
                   const int32_t* __restrict__ ids, bf16_t* __restrict__ yc, int R,
                   int64_t N, int per_wave) {
  constexpr int ROWB = 2 * E;                 // bytes of one field row
  constexpr int CR = ROWB / 16;               // 16-byte chunks per row
  constexpr int KPI = 1024 / ROWB;            // field rows per wave-wide DMA load
  constexpr int NI = NK / KPI;                // DMA loads per candidate
  constexpr int KS = NK / 16;                 // MFMA steps over fields
  constexpr int MB = E / 32;                  // 32-wide embedding blocks
  constexpr int O = 32 * NOB;                 // output fields
  constexpr int SO = O * ROWB;                // bytes of one candidate's output
  constexpr int NSO = SO / 1024;              // 1 KiB stores per candidate
  // A stage holds a candidate's input, then its output on the way out.
  constexpr int SB = NK * ROWB > SO ? NK * ROWB : SO;
  static_assert(NK % 16 == 0 && NK % KPI == 0 && (E == 64 || E == 128), "shape");
  static_assert(SO % 1024 == 0 && NI + NSO < 64, "output staging / vmcnt field");
  __shared__ __attribute__((aligned(1024))) char lds[kLcbWaves * kLcbStages * SB];
  ROCS_LDS char* const lds3 = (ROCS_LDS char*)lds;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int64_t first = ((int64_t)xcd_remap(blockIdx.x, gridDim.x) * kLcbWaves + wave) * per_wave;
  if (first >= N) return;
  const int count = (int)(N - first < per_wave ? N - first : per_wave);
  const uint32_t wbase = (uint32_t)(wave * kLcbStages * SB);   // this wave's ring (bytes)
  const uint32_t ring = lds_addr(lds) + wbase;

  // DMA lane map: load i fills rows KPI i + lane / CR, chunk position
  // lane % CR, taking chunk (lane % CR) ^ kv_swizzle(row) of that row.
  uint32_t soff[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int row = KPI * i + lane / CR;
    soff[i] = (uint32_t)(row * ROWB + 16 * ((lane % CR) ^ kv_swizzle<E>(row)));
  }
  auto issue = [&](int c) __attribute__((always_inline)) {
    const char* src = reinterpret_cast<const char*>(xc + (first + c) * (int64_t)(NK * E));
    const uint32_t dst = ring + (uint32_t)((c % kLcbStages) * SB);
#pragma unroll
    for (int i = 0; i < NI; ++i) lds_dma16_sv(src, soff[i], dst + (uint32_t)(KPI * i * ROWB));
  };

  // Transposing reads (as for V^T in the attention kernel): 16-lane group
  // g = lane / 16 reads rows 16 s + 4 (g / 2) + 8 rr + (lane % 16) / 4 and
  // columns 32 mb + 16 (g % 2) + 4 (lane % 4) .. +3; the mb step is an XOR
  // with 64 mb. Lane (l32, hh) then holds column 32 mb + l32 of fields
  // 16 s + 4 hh + {0..3} and 16 s + 8 + 4 hh + {0..3}.
  uint32_t ta[2];
#pragma unroll
  for (int rr = 0; rr < 2; ++rr) {
    const int g = lane >> 4, jl = lane & 15;
    const int row = 4 * (g >> 1) + 8 * rr + (jl >> 2);
    const int chunk0 = 2 * (g & 1) + ((jl & 3) >> 1);
    ta[rr] = (uint32_t)(row * ROWB + 16 * (chunk0 ^ kv_swizzle<E>(row)) + 8 * (jl & 1));
  }
  // B fragments: (W_CC)^T rows in the same field order, o = 32 ob + l32.
  bf16x8 wf[KS][NOB];
#pragma unroll
  for (int s = 0; s < KS; ++s)
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob) {
      const bf16_t* wr = wcc + (int64_t)(32 * ob + l32) * NK + 16 * s + 4 * hh;
      const u32x2 lo = *reinterpret_cast<const u32x2*>(wr);
      const u32x2 hi = *reinterpret_cast<const u32x2*>(wr + 8);
      wf[s][ob] = as_bf16x8(u32x4{lo[0], lo[1], hi[0], hi[1]});
    }

  // Request of the run's first candidate, then a forward walk.
  int r = -1;
  int64_t rend = 0;                 // first candidate past request r (CSR)
  if (ids == nullptr) {
    r = owner_of(off, R, first);
    rend = off[r + 1];
  }
  f32x16 zacc[MB][NOB];
  auto load_z = [&](int rq) __attribute__((always_inline)) {
    const float* zr = z + (int64_t)rq * O * E;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f32x4 v = *reinterpret_cast<const f32x4*>(
              zr + (int64_t)(32 * ob + l32) * E + 32 * mb + 8 * q + 4 * hh);
#pragma unroll
          for (int i = 0; i < 4; ++i) zacc[mb][ob][4 * q + i] = v[i];
        }
  };
  int zr_loaded = -1;

  issue(0);
  if (count > 1) issue(1);
  for (int c = 0; c < count; ++c) {
    const int64_t n = first + c;
    int rq;
    if (ids != nullptr) {
      rq = (int)min((uint32_t)ids[n], (uint32_t)(R - 1));
    } else {
      while (n >= rend && r + 1 < R) rend = off[++r + 1];   // bounded even for bad offsets
      rq = r;
    }
    if (rq != zr_loaded) {              // rare: a new request
      wait_vmcnt<0>();
      load_z(rq);
      zr_loaded = rq;
    }
    // Candidate c resident. Vector-memory operations retire in issue order,
    // so the wait allows exactly those issued after c's DMA loads: the
    // stores of c - 1 (c >= 1) and the loads of c + 1 (when there is a
    // c + 1). A smaller count would only wait longer; a larger one would not
    // make c resident.
    if (c >= 1) {
      if (c + 1 < count) wait_vmcnt<NSO + NI>(); else wait_vmcnt<NSO>();
    } else {
      if (count > 1) wait_vmcnt<NI>(); else wait_vmcnt<0>();
    }
    const uint32_t sbase = wbase + (uint32_t)((c % kLcbStages) * SB);
    f32x16 acc[MB][NOB];
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const uint32_t o = sbase + (uint32_t)(s * 16 * ROWB);
        const u32x2 lo = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (ROCS_LDS i16x4*)(lds3 + (o + (ta[0] ^ (64u * mb))))));
        const u32x2 hi = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (ROCS_LDS i16x4*)(lds3 + (o + (ta[1] ^ (64u * mb))))));
        const bf16x8 a = as_bf16x8(u32x4{lo[0], lo[1], hi[0], hi[1]});
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob)
          acc[mb][ob] = mfma32(a, wf[s][ob], s == 0 ? zacc[mb][ob] : acc[mb][ob]);
      }
    // Every transposing read of this stage has returned: it now takes the
    // output. Element 4 q + i of acc[mb][ob] is column 32 mb + 8 q + 4 hh + i
    // of output row 32 ob + l32; after the half-wave swap lane (l32, hh)
    // holds columns 32 mb + 16 j + 8 hh .. +7 (16-byte chunk 4 mb + 2 j + hh).
    __builtin_amdgcn_s_waitcnt((0 << 8) | (7 << 4) | 15 | (3 << 14));
    asm volatile("" ::: "memory");
    auto out_swz = [](int row) { return CR == 16 ? (row & 15) : ((row >> 1) & 7); };
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const f32x16& v = acc[mb][ob];
          const uint32_t e0 = pack_bf16x2(v[8 * j], v[8 * j + 1]);
          const uint32_t e1 = pack_bf16x2(v[8 * j + 2], v[8 * j + 3]);
          const uint32_t o0 = pack_bf16x2(v[8 * j + 4], v[8 * j + 5]);
          const uint32_t o1 = pack_bf16x2(v[8 * j + 6], v[8 * j + 7]);
          const auto s0 = __builtin_amdgcn_permlane32_swap(e0, o0, false, false);
          const auto s1 = __builtin_amdgcn_permlane32_swap(e1, o1, false, false);
          const int row = 32 * ob + l32;
          const int chunk = (4 * mb + 2 * j + hh) ^ out_swz(row);
          *reinterpret_cast<ROCS_LDS u32x4*>(lds3 + sbase + row * ROWB + 16 * chunk) =
              u32x4{s0[0], s1[0], s0[1], s1[1]};
        }
    // Read back row-contiguous: store i covers rows (1024 / ROWB) i .. , lane
    // -> row + lane / CR, chunk lane % CR; 1 KiB of contiguous output each.
    u32x4 ov[NSO];
#pragma unroll
    for (int i = 0; i < NSO; ++i) {
      const int row = (1024 / ROWB) * i + lane / CR;
      ov[i] = *reinterpret_cast<const ROCS_LDS u32x4*>(
          lds3 + sbase + row * ROWB + 16 * ((lane % CR) ^ out_swz(row)));
    }
    bf16_t* yr = yc + n * (int64_t)(O * E);
#pragma unroll
    for (int i = 0; i < NSO; ++i)
      *reinterpret_cast<u32x4*>(reinterpret_cast<char*>(yr) + 1024 * i + 16 * lane) = ov[i];
    // The stage is free once those reads have returned (the stores above
    // consumed them); the DMA of candidate c + 2 refills it.
    __builtin_amdgcn_s_waitcnt((0 << 8) | (7 << 4) | 15 | (3 << 14));
    asm volatile("" ::: "memory");
    if (c + 2 < count) issue(c + 2);
  }
}

// ---------------------------------------------------------------------------
// Request side, one launch for both request products (the stacked weight
// [W_RR; W_CR] applied to X^R_r): output row o < O_r goes to Y^R (input
// dtype), o >= O_r to Z (fp32, the candidate kernels' addend). One thread per
// output element; R is small next to N.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void lcb_request(
    const T* __restrict__ xr, const T* __restrict__ wrr, const T* __restrict__ wcr,
    T* __restrict__ yr, float* __restrict__ z, int R, int FR, int OR, int OC, int E) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t per_req = (int64_t)(OR + OC) * E;
  if (idx >= (int64_t)R * per_req) return;
  const int r = (int)(idx / per_req);
  const int o = (int)((idx % per_req) / E), e = (int)(idx % E);
  const bool req_out = o < OR;
  const T* w = req_out ? wrr + (int64_t)o * FR : wcr + (int64_t)(o - OR) * FR;
  const T* x = xr + (int64_t)r * FR * E + e;
  float acc = 0.f;
  for (int f = 0; f < FR; ++f) acc = fmaf(load_f32(w + f), load_f32(x + (int64_t)f * E), acc);
  if (req_out) yr[((int64_t)r * OR + o) * E + e] = from_f32<T>(acc);
  else z[((int64_t)r * OC + (o - OR)) * E + e] = acc;
}

// General candidate kernel (any F_c, O_c, E, dtype): one thread per output.
template <typename T>
__global__ __launch_bounds__(256) void lcb_cand_generic(
    const T* __restrict__ xc, const T* __restrict__ wcc, const float* __restrict__ z,
    const int32_t* __restrict__ off, const int32_t* __restrict__ ids, T* __restrict__ yc, int R,
    int64_t N, int FC, int OC, int E) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t per = (int64_t)OC * E;
  if (idx >= N * per) return;
  const int64_t n = idx / per;
  const int o = (int)((idx % per) / E), e = (int)(idx % E);
  const int r = ids != nullptr ? (int)min((uint32_t)ids[n], (uint32_t)(R - 1)) : owner_of(off, R, n);
  float acc = z[((int64_t)r * OC + o) * E + e];
  const T* x = xc + n * FC * E + e;
  for (int f = 0; f < FC; ++f)
    acc = fmaf(load_f32(wcc + (int64_t)o * FC + f), load_f32(x + (int64_t)f * E), acc);
  yc[idx] = from_f32<T>(acc);
}

template <int NK, int E, int NOB>
hipError_t launch_cand_fast(const LcbArgs& a, hipStream_t s) {
  int cus = 0;
  const hipError_t e = current_cu_count(&cus);
  if (e != hipSuccess) return e;
  // Runs of at least 4 candidates per wave, about eight waves per CU at once.
  const int64_t waves_target = (int64_t)cus * 8;
  int64_t per_wave = (a.N + waves_target - 1) / waves_target;
  per_wave = per_wave < 4 ? 4 : per_wave;
  const int64_t grid = (a.N + per_wave * kLcbWaves - 1) / (per_wave * kLcbWaves);
  return launch_kernel(lcb_cand_bf16<NK, E, NOB>, dim3((uint32_t)grid), dim3(64 * kLcbWaves), s,
                       static_cast<const bf16_t*>(a.x_cand), static_cast<const bf16_t*>(a.w_cc),
                       a.z, a.cand_offsets, a.ids, static_cast<bf16_t*>(a.y_cand), (int)a.R, a.N,
                       (int)per_wave);
}

template <int E, int NOB>
hipError_t dispatch_nk(const LcbArgs& a, hipStream_t s) {
  switch (a.f_cand) {
    case 16: return launch_cand_fast<16, E, NOB>(a, s);
    case 32: return launch_cand_fast<32, E, NOB>(a, s);
    default: return launch_cand_fast<64, E, NOB>(a, s);
  }
}

// Request side, bf16 with E a multiple of 4: each thread makes 4 adjacent
// embedding columns of one output row (8-byte input loads shared across the
// 4 columns, the weight row read once per field).
__global__ __launch_bounds__(256) void lcb_request_bf16x4(
    const bf16_t* __restrict__ xr, const bf16_t* __restrict__ wrr, const bf16_t* __restrict__ wcr,
    bf16_t* __restrict__ yr, float* __restrict__ z, int R, int FR, int OR, int OC, int E) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int E4 = E / 4;
  const int64_t per_req = (int64_t)(OR + OC) * E4;
  if (idx >= (int64_t)R * per_req) return;
  const int r = (int)(idx / per_req);
  const int o = (int)((idx % per_req) / E4), e = 4 * (int)(idx % E4);
  const bool req_out = o < OR;
  const bf16_t* w = req_out ? wrr + (int64_t)o * FR : wcr + (int64_t)(o - OR) * FR;
  const bf16_t* x = xr + (int64_t)r * FR * E + e;
  float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll 4
  for (int f = 0; f < FR; ++f) {
    const float wf = (float)w[f];
    const u32x2 v = *reinterpret_cast<const u32x2*>(x + (int64_t)f * E);
    a0 = fmaf(wf, bf16_lo(v[0]), a0);
    a1 = fmaf(wf, bf16_hi(v[0]), a1);
    a2 = fmaf(wf, bf16_lo(v[1]), a2);
    a3 = fmaf(wf, bf16_hi(v[1]), a3);
  }
  if (req_out) {
    *reinterpret_cast<u32x2*>(yr + ((int64_t)r * OR + o) * E + e) =
        u32x2{pack_bf16x2(a0, a1), pack_bf16x2(a2, a3)};
  } else {
    *reinterpret_cast<f32x4*>(z + ((int64_t)r * OC + (o - OR)) * E + e) = f32x4{a0, a1, a2, a3};
  }
}

template <typename T>
hipError_t launch_typed(const LcbArgs& a, bool fast, hipStream_t s) {
  hipError_t e;
  if (std::is_same_v<T, bf16_t> && fast) {
    // fast implies E in {64, 128} and 16-byte aligned rows
    const int64_t req_threads = a.R * (int64_t)(a.o_req + a.o_cand) * (a.emb / 4);
    if (!grid_fits((req_threads + 255) / 256, 256)) return hipErrorInvalidConfiguration;
    e = launch_kernel(lcb_request_bf16x4, dim3((uint32_t)((req_threads + 255) / 256)), dim3(256),
                      s, static_cast<const bf16_t*>(a.x_req), static_cast<const bf16_t*>(a.w_rr),
                      static_cast<const bf16_t*>(a.w_cr), static_cast<bf16_t*>(a.y_req), a.z,
                      (int)a.R, a.f_req, a.o_req, a.o_cand, a.emb);
  } else {
    const int64_t req_elems = a.R * (int64_t)(a.o_req + a.o_cand) * a.emb;
    if (!grid_fits((req_elems + 255) / 256, 256)) return hipErrorInvalidConfiguration;
    e = launch_kernel(lcb_request<T>, dim3((uint32_t)((req_elems + 255) / 256)), dim3(256),
                      s, static_cast<const T*>(a.x_req), static_cast<const T*>(a.w_rr),
                      static_cast<const T*>(a.w_cr), static_cast<T*>(a.y_req), a.z,
                      (int)a.R, a.f_req, a.o_req, a.o_cand, a.emb);
  }
  if (e != hipSuccess || a.N == 0) return e;
  if constexpr (std::is_same_v<T, bf16_t>) {
    if (fast) {
      if (a.emb == 128) return dispatch_nk<128, 1>(a, s);
      return a.o_cand == 64 ? dispatch_nk<64, 2>(a, s) : dispatch_nk<64, 1>(a, s);
    }
  }
  const int64_t cand_elems = a.N * (int64_t)a.o_cand * a.emb;
  if (!grid_fits((cand_elems + 255) / 256, 256)) return hipErrorInvalidConfiguration;
  return launch_kernel(lcb_cand_generic<T>, dim3((uint32_t)((cand_elems + 255) / 256)), dim3(256),
                       s, static_cast<const T*>(a.x_cand), static_cast<const T*>(a.w_cc), a.z,
                       a.cand_offsets, a.ids, static_cast<T*>(a.y_cand), (int)a.R, a.N, a.f_cand,
                       a.o_cand, a.emb);
}

}  // namespace

bool lcb_fast_shape(int f_cand, int o_cand, int emb) {
  return (f_cand == 16 || f_cand == 32 || f_cand == 64) &&
         ((emb == 128 && o_cand == 32) || (emb == 64 && (o_cand == 32 || o_cand == 64)));
}

hipError_t launch_lcb(const LcbArgs& a, bool fast, hipStream_t s) {
  return a.bf16 ? launch_typed<bf16_t>(a, fast, s) : launch_typed<float>(a, fast, s);
}

}  // namespace rocs
