// GLM-masked factorization machine, two groups (Eq. glm-fm, Eq. glm-fm-two-groups).
//
//   Y^R_r = X^R_r (X^R_r)^T                         once per request
//   Y^C_n = [ X^C_n (X^R_{m_n})^T | X^C_n (X^C_n)^T ]  per candidate
//
// IKBO form: a workgroup owns a tile of one request's candidates, so the
// request's field embeddings X^R_r are the shared MFMA operand of every
// candidate in the tile (read once per tile, never copied per candidate). The
// request-only block Y^R is produced by the request's first tile slot, so
// requests without candidates still get it. The masked request-row /
// candidate-column block is never computed.
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace rocs {
namespace {

constexpr int kFmRows = 256;   // candidate-field rows per workgroup (4 waves x 64)

// ---------------------------------------------------------------------------
// bf16 MFMA kernel: f_req multiple of 16, f_cand FC in {4, 8, 16}, emb
// multiple of 32. Candidate-field rows are the flattened [N * FC, E] view.
// Products (A, B roles chosen so each lane ends with 4 consecutive output
// columns of one output row, written as one 8-byte store):
//   request-candidate: C[j][row] = <x^R_j, x^C_row>     (A = X^R, B = X^C)
//   candidate-candidate: C[row'][row] within a 16-row block (A = B = X^C);
//     only pairs from the same candidate are kept (FC divides 16).
//   request-request: C[j'][i] = <x^R_j', x^R_i> = Y^R[i][j'].
// ---------------------------------------------------------------------------
template <int FC>
__global__ __launch_bounds__(256) void glm_fm_bf16(
    const bf16_t* __restrict__ xr, const bf16_t* __restrict__ xc,
    const int32_t* __restrict__ off, bf16_t* __restrict__ yr, bf16_t* __restrict__ yc, int R,
    int FR, int E) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, g = lane >> 4;
  const uint32_t slot = xcd_remap(blockIdx.x, gridDim.x);
  const int r = request_of_slot(off, R, slot, FC, kFmRows);
  const int64_t j = (int64_t)slot - tile_base(off, r, FC, kFmRows);
  const int64_t rbeg = (int64_t)off[r] * FC, rend = (int64_t)off[r + 1] * FC;
  const bf16_t* xrr = xr + (int64_t)r * FR * E;
  const int KS = E / 32, JB = FR / 16;

  if (j == 0 && yr != nullptr) {
    bf16_t* yrr = yr + (int64_t)r * FR * FR;
    for (int b = wave; b < JB * JB; b += 4) {
      const int ib = b / JB, jb = b % JB;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 a = as_bf16x8(load16(xrr + (16 * jb + lr) * E + 32 * ks + 8 * g, true));
        const bf16x8 bb = as_bf16x8(load16(xrr + (16 * ib + lr) * E + 32 * ks + 8 * g, true));
        acc = mfma16(a, bb, acc);
      }
      // acc[i] = Y^R[16 ib + lr][16 jb + 4 g + i]
      *reinterpret_cast<u32x2*>(yrr + (16 * ib + lr) * FR + 16 * jb + 4 * g) =
          u32x2{pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3])};
    }
  }
  const int64_t row0 = rbeg + j * kFmRows;
  if (yc == nullptr || row0 >= rend) return;
  const int rows = (int)(rend - row0 < kFmRows ? rend - row0 : kFmRows);
  const int ystride = FC * (FR + FC);          // y_cand row length
  for (int rb = 0; rb < 4; ++rb) {
    const int rr = wave * 64 + 16 * rb;         // first row of this 16-row block
    if (rr >= rows) break;
    const int row = rr + lr;
    const bool ok = row < rows;
    const int64_t grow = row0 + row;            // = n * FC + fi
    const bf16_t* xcr = xc + grow * E;
    f32x4 cc = {0.f, 0.f, 0.f, 0.f};
    // request-candidate block, 16 request fields at a time
    for (int jb = 0; jb < JB; ++jb) {
      f32x4 rc = {0.f, 0.f, 0.f, 0.f};
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 b = as_bf16x8(load16(xcr + 32 * ks + 8 * g, ok));
        const bf16x8 a = as_bf16x8(load16(xrr + (16 * jb + lr) * E + 32 * ks + 8 * g, true));
        rc = mfma16(a, b, rc);
        if (jb == 0) cc = mfma16(b, b, cc);
      }
      // rc[i] = <x^R_{16 jb + 4 g + i}, x^C_row>
      if (ok) {
        const int64_t n = grow / FC, fi = grow % FC;
        *reinterpret_cast<u32x2*>(yc + n * ystride + fi * (FR + FC) + 16 * jb + 4 * g) =
            u32x2{pack_bf16x2(rc[0], rc[1]), pack_bf16x2(rc[2], rc[3])};
      }
    }
    // cc[i] = <x^C_{rr + 4 g + i}, x^C_row>; same candidate iff (4 g) / FC == lr / FC.
    if (ok && (4 * g) / FC == lr / FC) {
      const int64_t n = grow / FC, fi = grow % FC;
      *reinterpret_cast<u32x2*>(yc + n * ystride + fi * (FR + FC) + FR + (4 * g) % FC) =
          u32x2{pack_bf16x2(cc[0], cc[1]), pack_bf16x2(cc[2], cc[3])};
    }
  }
}

// ---------------------------------------------------------------------------
// General kernels: any dtype and sizes; one thread per output value.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void glm_fm_request_generic(const T* __restrict__ xr,
                                                              T* __restrict__ yr, int64_t R,
                                                              int FR, int E) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= R * FR * FR) return;
  const int64_t r = idx / ((int64_t)FR * FR);
  const int i = (int)(idx / FR % FR), jj = (int)(idx % FR);
  const T* a = xr + (r * FR + i) * E;
  const T* b = xr + (r * FR + jj) * E;
  float acc = 0.f;
  for (int e = 0; e < E; ++e) acc = fmaf(load_f32(a + e), load_f32(b + e), acc);
  yr[idx] = from_f32<T>(acc);
}

template <typename T>
__global__ __launch_bounds__(256) void glm_fm_cand_generic(const T* __restrict__ xr,
                                                           const T* __restrict__ xc,
                                                           const int32_t* __restrict__ off,
                                                           T* __restrict__ yc, int R, int64_t N,
                                                           int FR, int FC, int E) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int width = FR + FC;
  if (idx >= N * FC * width) return;
  const int64_t n = idx / ((int64_t)FC * width);
  const int fi = (int)(idx / width % FC), col = (int)(idx % width);
  const T* a = xc + (n * FC + fi) * E;
  const T* b = col < FR ? xr + ((int64_t)owner_of(off, R, n) * FR + col) * E
                        : xc + (n * FC + (col - FR)) * E;
  float acc = 0.f;
  for (int e = 0; e < E; ++e) acc = fmaf(load_f32(a + e), load_f32(b + e), acc);
  yc[idx] = from_f32<T>(acc);
}

template <int FC>
hipError_t launch_fast(const InteractionArgs& a, hipStream_t s) {
  const int64_t slots = a.R + (a.N * FC + kFmRows - 1) / kFmRows;
  if (!grid_fits(slots, 256)) return hipErrorInvalidConfiguration;
  return launch_kernel(glm_fm_bf16<FC>, dim3((uint32_t)slots), dim3(256), s,
                       static_cast<const bf16_t*>(a.x_req), static_cast<const bf16_t*>(a.x_cand),
                       a.cand_offsets, static_cast<bf16_t*>(a.y_req),
                       static_cast<bf16_t*>(a.y_cand), (int)a.R, a.f_req, a.emb);
}

template <typename T>
hipError_t launch_generic(const InteractionArgs& a, hipStream_t s) {
  hipError_t e = hipSuccess;
  if (a.y_req != nullptr) {
    const int64_t n = a.R * a.f_req * a.f_req;
    if (!grid_fits((n + 255) / 256, 256)) return hipErrorInvalidConfiguration;
    e = launch_kernel(glm_fm_request_generic<T>, dim3((uint32_t)((n + 255) / 256)), dim3(256), s,
                      static_cast<const T*>(a.x_req), static_cast<T*>(a.y_req), a.R, a.f_req,
                      a.emb);
    if (e != hipSuccess) return e;
  }
  if (a.y_cand != nullptr && a.N > 0) {
    const int64_t n = a.N * a.f_cand * (a.f_req + a.f_cand);
    if (!grid_fits((n + 255) / 256, 256)) return hipErrorInvalidConfiguration;
    e = launch_kernel(glm_fm_cand_generic<T>, dim3((uint32_t)((n + 255) / 256)), dim3(256), s,
                      static_cast<const T*>(a.x_req), static_cast<const T*>(a.x_cand),
                      a.cand_offsets, static_cast<T*>(a.y_cand), (int)a.R, a.N, a.f_req,
                      a.f_cand, a.emb);
  }
  return e;
}

}  // namespace

hipError_t launch_interaction(const InteractionArgs& a, bool fast, hipStream_t s) {
  if (!fast) return a.bf16 ? launch_generic<bf16_t>(a, s) : launch_generic<float>(a, s);
  switch (a.f_cand) {
    case 4: return launch_fast<4>(a, s);
    case 8: return launch_fast<8>(a, s);
    default: return launch_fast<16>(a, s);
  }
}

}  // namespace rocs
