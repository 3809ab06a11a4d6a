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
// Request-side GEMM, bf16 in, fp32 Z out. One workgroup per 16 x 16 tile of
// Z; its four waves split K in 32-wide steps (operands straight from global
// memory into MFMA registers, each lane's 8 consecutive k are one 16-byte
// load) and reduce through LDS in a fixed order. Workgroups past the Z tiles
// expand the index map.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void request_gemm_bf16(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ w, float* __restrict__ z,
    const int32_t* __restrict__ off, int32_t* __restrict__ ids, int R, int64_t N, int K, int D,
    int tiles_d, int z_blocks) {
  const int tid = threadIdx.x;
  if ((int)blockIdx.x >= z_blocks) {
    const int64_t n = (int64_t)(blockIdx.x - z_blocks) * 256 + tid;
    if (n < N) ids[n] = owner_of(off, R, n);
    return;
  }
  __shared__ f32x4 red[4][kWave];
  const int lane = tid & 63, wave = tid >> 6;
  const int r0 = ((int)blockIdx.x / tiles_d) * 16, d0 = ((int)blockIdx.x % tiles_d) * 16;
  const int row = lane & 15, kq = (lane >> 4) * 8;
  const bool dok = d0 + row < D, rok = r0 + row < R;
  const bf16_t* wp = w + (int64_t)(d0 + row) * K + kq;
  const bf16_t* xp = x + (int64_t)(r0 + row) * K + kq;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int k = wave * 32; k < K; k += 128) {
    const bool kok = k + kq < K;
    const bf16x8 a = as_bf16x8(load16(wp + k, dok && kok));
    const bf16x8 b = as_bf16x8(load16(xp + k, rok && kok));
    acc = mfma16(a, b, acc);   // acc[i] = Z[r0 + row][d0 + 4 (lane / 16) + i]
  }
  red[wave][lane] = acc;
  __syncthreads();
  if (wave == 0) {
    const f32x4 s = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
    const int d = d0 + (lane >> 4) * 4;
    if (rok && d < D) *reinterpret_cast<f32x4*>(z + (int64_t)(r0 + row) * D + d) = s;
  }
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
    bf16_t* __restrict__ out, int64_t N, int K, int D, int tiles_m, int relu) {
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
    const bool one_request = z != nullptr && ids[n0] == ids[(n0 + BN < N ? n0 + BN : N) - 1];
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int64_t n = n0 + wn0 + 32 * fn + l32;
      const float* zr = nullptr;
      if (z != nullptr) {
        const int r = one_request ? ids[n0] : (n < N ? ids[n] : 0);
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
    T* __restrict__ out, int64_t N, int K, int D, int relu) {
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
  if (z != nullptr) acc += z[(int64_t)ids[n] * D + d];
  if (bias != nullptr) acc += bias[d];
  if (relu) acc = fmaxf(acc, 0.f);
  out[idx] = from_f32<T>(acc);
}

template <int BM, int BN, int BK, int WMW, int WNW>
hipError_t launch_fast_gemm(const LinearArgs& a, hipStream_t s) {
  const int tiles_m = (int)((a.d_out + BM - 1) / BM);
  const int64_t tiles_n = (a.N + BN - 1) / BN;
  const int64_t grid = tiles_m * tiles_n;
  const bf16_t* x = static_cast<const bf16_t*>(a.x_cand);
  const bf16_t* xa = static_cast<const bf16_t*>(a.x_cand_add);
  const bf16_t* w = static_cast<const bf16_t*>(a.w_cand);
  bf16_t* o = static_cast<bf16_t*>(a.out);
  const float* z = a.k_req > 0 ? a.z : nullptr;
  if (xa != nullptr)
    return launch_kernel(ikbo_gemm_bf16<BM, BN, BK, WMW, WNW, true>, dim3((uint32_t)grid),
                         dim3(64 * WMW * WNW), s,
                         x, xa, w, a.bias, z, a.ids, o, a.N, (int)a.k_cand, (int)a.d_out,
                         tiles_m, (int)a.relu);
  return launch_kernel(ikbo_gemm_bf16<BM, BN, BK, WMW, WNW, false>, dim3((uint32_t)grid),
                       dim3(64 * WMW * WNW), s,
                       x, xa, w, a.bias, z, a.ids, o, a.N, (int)a.k_cand, (int)a.d_out,
                       tiles_m, (int)a.relu);
}

template <typename T>
hipError_t launch_generic(const LinearArgs& a, hipStream_t s) {
  hipError_t e = hipSuccess;
  if (a.k_req > 0) {
    const int z_blocks = (int)((a.R * a.d_out + 255) / 256);
    const int id_blocks = (int)((a.N + 255) / 256);
    e = launch_kernel(request_gemm_generic<T>, dim3(z_blocks + id_blocks), dim3(256), s,
                      static_cast<const T*>(a.x_req), static_cast<const T*>(a.w_req), a.z,
                      a.cand_offsets, a.ids, (int)a.R, a.N, (int)a.k_req, (int)a.d_out,
                      z_blocks);
    if (e != hipSuccess) return e;
  }
  const int64_t blocks = (a.N * a.d_out + 255) / 256;
  return launch_kernel(linear_generic<T>, dim3((uint32_t)blocks), dim3(256), s,
                       static_cast<const T*>(a.x_cand), static_cast<const T*>(a.x_cand_add),
                       static_cast<const T*>(a.w_cand), a.bias,
                       a.k_req > 0 ? a.z : nullptr, a.ids, static_cast<T*>(a.out), a.N,
                       (int)a.k_cand, (int)a.d_out, (int)a.relu);
}

}  // namespace

hipError_t launch_request_ids(const int32_t* off, int64_t R, int64_t N, int32_t* ids,
                              hipStream_t s) {
  return launch_kernel(request_ids_kernel, dim3((uint32_t)((N + 255) / 256)), dim3(256), s,
                       off, (int)R, N, ids);
}

hipError_t launch_linear(const LinearArgs& a, bool fast, hipStream_t s) {
  if (!fast) return a.bf16 ? launch_generic<bf16_t>(a, s) : launch_generic<float>(a, s);
  if (a.k_req > 0) {
    const int tiles_d = (int)((a.d_out + 15) / 16);
    const int z_blocks = tiles_d * (int)((a.R + 15) / 16);
    const int id_blocks = (int)((a.N + 255) / 256);
    hipError_t e = launch_kernel(request_gemm_bf16, dim3(z_blocks + id_blocks), dim3(256), s,
                                 static_cast<const bf16_t*>(a.x_req),
                                 static_cast<const bf16_t*>(a.w_req), a.z, a.cand_offsets,
                                 a.ids, (int)a.R, a.N, (int)a.k_req, (int)a.d_out, tiles_d,
                                 z_blocks);
    if (e != hipSuccess) return e;
  }
  // Large tiles when they still give every CU at least four tiles.
  const int64_t big_tiles = ((a.d_out + 255) / 256) * ((a.N + 127) / 128);
  if (big_tiles >= 1024) return launch_fast_gemm<256, 128, 32, 2, 2>(a, s);
  return launch_fast_gemm<128, 128, 32, 2, 2>(a, s);
}

}  // namespace rocs
