// C ABI of librocs: argument validation, fast-path selection, error reporting.
// Nothing here touches tensor data; every operation runs in the kernels.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/rocs.h"
#include "kernels.h"

namespace {

thread_local std::string g_error;

int32_t fail(rocs_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_error = buf;
  return s;
}

int32_t ok() {
  g_error.clear();
  return ROCS_OK;
}

// A launcher's error: a grid too large for one launch (the launchers test
// their computed grids before narrowing them) is a shape this build does not
// run; anything else is the runtime's refusal.
int32_t launch_failed(const char* name, hipError_t e) {
  if (e == hipErrorInvalidConfiguration)
    return fail(ROCS_ERR_UNSUPPORTED, "%s: the launch grid would exceed 2^32 work items", name);
  return fail(ROCS_ERR_HIP, "%s: %s", name, hipGetErrorString(e));
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// Byte ranges [a, a + an) and [b, b + bn) intersect.
bool overlap(const void* a, size_t an, const void* b, size_t bn) {
  if (a == nullptr || b == nullptr || an == 0 || bn == 0) return false;
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + bn && y < x + an;
}

size_t align256(size_t n) { return (n + 255) & ~size_t(255); }

bool valid_dtype(int32_t d) { return d == ROCS_DTYPE_F32 || d == ROCS_DTYPE_BF16; }
size_t esize(int32_t d) { return d == ROCS_DTYPE_BF16 ? 2 : 4; }

constexpr int64_t kMaxI32 = 2147483647;

}  // namespace

extern "C" {

int32_t rocs_abi_version(void) { return ROCS_ABI_VERSION; }

const char* rocs_status_string(int32_t s) {
  switch (s) {
    case ROCS_OK: return "ok";
    case ROCS_ERR_INVALID_ARGUMENT: return "invalid argument";
    case ROCS_ERR_UNSUPPORTED: return "unsupported";
    case ROCS_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case ROCS_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* rocs_last_error_message(void) { return g_error.c_str(); }

size_t rocs_ikbo_linear_workspace_size(int64_t num_requests, int64_t num_cand, int64_t d_out,
                                       int64_t k_req) {
  if (k_req <= 0 || num_requests <= 0 || num_cand <= 0 || d_out <= 0) return 0;
  // Request table Z [R, d_out] fp32, then one region that holds either the
  // expanded index map [N] int32 or the combined kernel's completion flags
  // (one 64-bit word per 16 x 16 tile of Z).
  const size_t ids = (size_t)num_cand * sizeof(int32_t);
  const size_t flags = (size_t)((num_requests + 15) / 16) * (size_t)((d_out + 15) / 16) * 8;
  return align256((size_t)num_requests * (size_t)d_out * sizeof(float)) +
         align256(ids > flags ? ids : flags);
}

}  // extern "C"

namespace {

// Shared by rocs_ikbo_linear (CSR offsets) and rocs_ikbo_linear_mapped (a
// per-candidate request map, `mapped`): only one of cand_offsets / cand_ids
// is read.
struct RequestSide {          // full GLM layer: Y^R = act(x_req W_RR^T + b^R)
  const void* w_rr = nullptr;
  const float* b_rr = nullptr;
  void* y_req = nullptr;
  int64_t d_req = 0;
};

int32_t linear_impl(const char* name, bool mapped, const void* x_req, int64_t k_req,
                    const void* x_cand, const void* x_cand_add, int64_t k_cand,
                    const void* w_req, const void* w_cand, const float* bias,
                    const int32_t* cand_offsets, const int32_t* cand_ids, int64_t R, int64_t N,
                    int64_t d_out, int32_t dtype, int32_t activation, void* out,
                    void* workspace, size_t workspace_bytes, void* stream,
                    const RequestSide& rs = RequestSide(), bool combined = false) {
  const bool full = rs.y_req != nullptr;
  if (!valid_dtype(dtype)) return fail(ROCS_ERR_INVALID_ARGUMENT, "unknown dtype %d", dtype);
  if (activation != ROCS_ACT_NONE && activation != ROCS_ACT_RELU)
    return fail(ROCS_ERR_INVALID_ARGUMENT, "unknown activation %d", activation);
  if (R < 0 || N < 0 || k_req < 0 || k_cand < 1 || d_out < 1)
    return fail(ROCS_ERR_INVALID_ARGUMENT,
                "sizes must satisfy R >= 0, N >= 0, k_req >= 0, k_cand >= 1, d_out >= 1 "
                "(got R=%lld N=%lld k_req=%lld k_cand=%lld d_out=%lld)",
                (long long)R, (long long)N, (long long)k_req, (long long)k_cand,
                (long long)d_out);
  if (N > kMaxI32 || R > kMaxI32 || k_req > kMaxI32 || k_cand > kMaxI32 || d_out > kMaxI32 ||
      rs.d_req > kMaxI32)
    return fail(ROCS_ERR_UNSUPPORTED, "a size exceeds 2^31 - 1");
  if (full) {
    if (k_req < 1 || rs.d_req < 1 || rs.w_rr == nullptr || x_req == nullptr)
      return fail(ROCS_ERR_INVALID_ARGUMENT,
                  "the request-side output needs k_req >= 1, d_req >= 1, x_req and w_rr");
    if (R == 0 && N == 0) return ok();
  } else if (N == 0) {
    return ok();
  }
  if (k_req > 0 && R == 0)
    return fail(ROCS_ERR_INVALID_ARGUMENT, "N > 0 candidates but no requests to own them");
  if (N > 0 && (x_cand == nullptr || w_cand == nullptr || out == nullptr))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "x_cand, w_cand and out must not be NULL");
  if (k_req > 0 && (x_req == nullptr || w_req == nullptr ||
                    (mapped ? cand_ids == nullptr : cand_offsets == nullptr)))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "k_req > 0 needs x_req, w_req and %s",
                mapped ? "cand_request_ids" : "cand_offsets");
  const size_t need = rocs_ikbo_linear_workspace_size(R, N, d_out, k_req);
  if (need > 0) {
    if (workspace == nullptr || workspace_bytes < need)
      return fail(ROCS_ERR_WORKSPACE_TOO_SMALL, "workspace needs %zu bytes, got %zu", need,
                  workspace == nullptr ? (size_t)0 : workspace_bytes);
    if (!aligned(workspace, 256))
      return fail(ROCS_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  }
  const size_t es = esize(dtype);
  const size_t out_bytes = (size_t)N * d_out * es;
  const struct { const void* p; size_t n; const char* name; } ins[] = {
      {x_req, (size_t)R * k_req * es, "x_req"},
      {x_cand, (size_t)N * k_cand * es, "x_cand"},
      {x_cand_add, (size_t)N * k_cand * es, "x_cand_add"},
      {w_req, (size_t)d_out * k_req * es, "w_req"},
      {w_cand, (size_t)d_out * k_cand * es, "w_cand"},
      {bias, (size_t)d_out * sizeof(float), "bias"},
      {cand_offsets, (size_t)(R + 1) * sizeof(int32_t), "cand_offsets"},
      {cand_ids, (size_t)N * sizeof(int32_t), "cand_request_ids"},
      {need > 0 ? workspace : nullptr, need, "workspace"},
  };
  const size_t yr_bytes = full ? (size_t)R * rs.d_req * es : 0;
  for (const auto& in : ins) {
    if (overlap(out, out_bytes, in.p, in.n))
      return fail(ROCS_ERR_INVALID_ARGUMENT, "out overlaps %s", in.name);
    if (overlap(rs.y_req, yr_bytes, in.p, in.n))
      return fail(ROCS_ERR_INVALID_ARGUMENT, "y_req overlaps %s", in.name);
  }
  if (full && (overlap(rs.y_req, yr_bytes, out, out_bytes) ||
               overlap(rs.y_req, yr_bytes, rs.w_rr, (size_t)rs.d_req * k_req * es) ||
               overlap(rs.y_req, yr_bytes, rs.b_rr, (size_t)rs.d_req * sizeof(float)) ||
               overlap(out, out_bytes, rs.w_rr, (size_t)rs.d_req * k_req * es) ||
               overlap(out, out_bytes, rs.b_rr, (size_t)rs.d_req * sizeof(float))))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "y_req overlaps out or the W_RR / b^R inputs");
  if (need > 0) {
    const size_t zb = align256((size_t)R * d_out * sizeof(float));
    const struct { const void* p; size_t n; const char* name; } inw[] = {
        {x_req, (size_t)R * k_req * es, "x_req"}, {x_cand, (size_t)N * k_cand * es, "x_cand"},
        {w_req, (size_t)d_out * k_req * es, "w_req"}, {w_cand, (size_t)d_out * k_cand * es, "w_cand"},
        {cand_offsets, (size_t)(R + 1) * sizeof(int32_t), "cand_offsets"},
        {cand_ids, (size_t)N * sizeof(int32_t), "cand_request_ids"},
        {rs.y_req, (size_t)R * rs.d_req * es, "y_req"}};
    for (const auto& in : inw)
      if (overlap(workspace, need, in.p, in.n))
        return fail(ROCS_ERR_INVALID_ARGUMENT, "workspace overlaps %s", in.name);
    (void)zb;
  }

  rocs::LinearArgs a{};
  a.x_req = x_req; a.x_cand = x_cand; a.x_cand_add = x_cand_add;
  a.w_req = w_req; a.w_cand = w_cand; a.bias = bias; a.cand_offsets = cand_offsets;
  a.R = R; a.N = N; a.k_req = k_req; a.k_cand = k_cand; a.d_out = d_out;
  a.bf16 = dtype == ROCS_DTYPE_BF16;
  a.relu = activation == ROCS_ACT_RELU;
  a.out = out;
  a.w_rr = rs.w_rr; a.b_rr = rs.b_rr; a.y_req = rs.y_req; a.d_req = rs.d_req;
  a.combined = combined;
  if (need > 0) {
    a.z = static_cast<float*>(workspace);
    a.ids = mapped ? const_cast<int32_t*>(cand_ids)
                   : reinterpret_cast<int32_t*>(static_cast<char*>(workspace) +
                                                align256((size_t)R * d_out * sizeof(float)));
    a.ids_given = mapped;
  }
  const bool fast = a.bf16 && k_cand % 8 == 0 && k_req % 8 == 0 && d_out % 4 == 0 &&
                    aligned(x_cand, 16) && aligned(x_cand_add, 16) && aligned(w_cand, 16) &&
                    aligned(x_req, 16) && aligned(w_req, 16) && aligned(bias, 16) &&
                    aligned(out, 16) &&
                    (!full || (rs.d_req % 4 == 0 && aligned(rs.w_rr, 16) &&
                               aligned(rs.b_rr, 16) && aligned(rs.y_req, 8)));
  // The general kernels run one thread per output element (and the request
  // kernel one per request-side element); keep their grids under 2^32 items.
  if (!fast && ((N * d_out) >> 32 != 0 || (R * (d_out + (full ? rs.d_req : 0))) >> 32 != 0 ||
                (full && (R * rs.d_req) >> 32 != 0)))
    return fail(ROCS_ERR_UNSUPPORTED, "%s: the general kernel's grid would exceed 2^32 threads "
                "(N * d_out = %lld); the bf16 fast path has no such limit", name,
                (long long)(N * d_out));
  const hipError_t e = rocs::launch_linear(a, fast, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return launch_failed(name, e);
  return ok();
}

}  // namespace

extern "C" {

int32_t rocs_ikbo_linear(const void* x_req, int64_t k_req, const void* x_cand,
                         const void* x_cand_add, int64_t k_cand, const void* w_req,
                         const void* w_cand, const float* bias, const int32_t* cand_offsets,
                         int64_t R, int64_t N, int64_t d_out, int32_t dtype, int32_t activation,
                         void* out, void* workspace, size_t workspace_bytes, void* stream) {
  return linear_impl("rocs_ikbo_linear", false, x_req, k_req, x_cand, x_cand_add, k_cand,
                     w_req, w_cand, bias, cand_offsets, nullptr, R, N, d_out, dtype, activation,
                     out, workspace, workspace_bytes, stream);
}

int32_t rocs_glm_linear(const void* x_req, int64_t k_req, const void* x_cand,
                        const void* x_cand_add, int64_t k_cand, const void* w_rr,
                        const void* w_cr, const void* w_cc, const float* b_req,
                        const float* b_cand, const int32_t* cand_offsets, int64_t R, int64_t N,
                        int64_t d_req, int64_t d_cand, int32_t dtype, int32_t activation,
                        void* y_req, void* y_cand, void* workspace, size_t workspace_bytes,
                        void* stream) {
  if (y_req == nullptr) return fail(ROCS_ERR_INVALID_ARGUMENT, "y_req must not be NULL");
  RequestSide rs;
  rs.w_rr = w_rr; rs.b_rr = b_req; rs.y_req = y_req; rs.d_req = d_req;
  return linear_impl("rocs_glm_linear", false, x_req, k_req, x_cand, x_cand_add, k_cand, w_cr,
                     w_cc, b_cand, cand_offsets, nullptr, R, N, d_cand, dtype, activation,
                     y_cand, workspace, workspace_bytes, stream, rs);
}

int32_t rocs_ikbo_linear_combined(const void* x_req, int64_t k_req, const void* x_cand,
                                  const void* x_cand_add, int64_t k_cand, const void* w_rr,
                                  const void* w_cr, const void* w_cc, const float* b_req,
                                  const float* b_cand, const int32_t* cand_offsets, int64_t R,
                                  int64_t N, int64_t d_req, int64_t d_cand, int32_t dtype,
                                  int32_t activation, void* y_req, void* y_cand,
                                  void* workspace, size_t workspace_bytes, void* stream) {
  RequestSide rs;
  if (y_req != nullptr) {
    rs.w_rr = w_rr; rs.b_rr = b_req; rs.y_req = y_req; rs.d_req = d_req;
  }
  return linear_impl("rocs_ikbo_linear_combined", false, x_req, k_req, x_cand, x_cand_add,
                     k_cand, w_cr, w_cc, b_cand, cand_offsets, nullptr, R, N, d_cand, dtype,
                     activation, y_cand, workspace, workspace_bytes, stream, rs, true);
}

}  // extern "C"

namespace {

// Scratch of rocs_ikbo_linear_noalloc: the request table Z and the index map
// live in this array instead of a caller's workspace. Each device that runs
// the library holds its own copy until the process ends. In host code the
// name only stands in for the symbol; the device address comes from
// hipGetSymbolAddress, taken once per device with that device current.
constexpr size_t kScratchBytes = ROCS_NOALLOC_SCRATCH_BYTES;
static __device__ __attribute__((aligned(256))) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
struct ScratchSlot {
  std::once_flag once;
  void* ptr = nullptr;
  hipError_t err = hipSuccess;
};
ScratchSlot g_scratch[kMaxDevices];

// The current device's copy of `scratch` (its device address).
hipError_t scratch_address(void** out) {
  int dev = 0;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  ScratchSlot& slot = g_scratch[dev];
  std::call_once(slot.once, [&slot] {
    slot.err = hipGetSymbolAddress(&slot.ptr, HIP_SYMBOL(scratch));
  });
  if (slot.err != hipSuccess) return slot.err;
  *out = slot.ptr;
  return hipSuccess;
}

}  // namespace

extern "C" {

int32_t rocs_ikbo_linear_noalloc(const void* x_req, int64_t k_req, const void* x_cand,
                                 const void* x_cand_add, int64_t k_cand, const void* w_req,
                                 const void* w_cand, const float* bias,
                                 const int32_t* cand_offsets, int64_t R, int64_t N,
                                 int64_t d_out, int32_t dtype, int32_t activation, void* out,
                                 void* stream) {
  // Size first, before any HIP call: the request table and the index map
  // must fit the static scratch array.
  const size_t need = rocs_ikbo_linear_workspace_size(R, N, d_out, k_req);
  if (need > kScratchBytes)
    return fail(ROCS_ERR_WORKSPACE_TOO_SMALL,
                "rocs_ikbo_linear_noalloc: needs %zu bytes of scratch for R=%lld N=%lld "
                "d_out=%lld; the library's static scratch holds %zu (use rocs_ikbo_linear "
                "with a workspace)", need, (long long)R, (long long)N, (long long)d_out,
                kScratchBytes);
  void* ws = nullptr;
  if (need > 0 && N > 0) {
    const hipError_t e = scratch_address(&ws);
    if (e != hipSuccess)
      return fail(ROCS_ERR_HIP, "rocs_ikbo_linear_noalloc: scratch address: %s",
                  hipGetErrorString(e));
  }
  return linear_impl("rocs_ikbo_linear_noalloc", false, x_req, k_req, x_cand, x_cand_add,
                     k_cand, w_req, w_cand, bias, cand_offsets, nullptr, R, N, d_out, dtype,
                     activation, out, ws, ws != nullptr ? kScratchBytes : 0, stream);
}

int32_t rocs_ikbo_linear_mapped(const void* x_req, int64_t k_req, const void* x_cand,
                                const void* x_cand_add, int64_t k_cand, const void* w_req,
                                const void* w_cand, const float* bias,
                                const int32_t* cand_request_ids, int64_t R, int64_t N,
                                int64_t d_out, int32_t dtype, int32_t activation, void* out,
                                void* workspace, size_t workspace_bytes, void* stream) {
  return linear_impl("rocs_ikbo_linear_mapped", true, x_req, k_req, x_cand, x_cand_add,
                     k_cand, w_req, w_cand, bias, nullptr, cand_request_ids, R, N, d_out, dtype,
                     activation, out, workspace, workspace_bytes, stream);
}

}  // extern "C"

namespace {

// Shared by rocs_dca_attention (CSR cand_offsets) and rocs_dca_attention_mapped
// (a per-candidate request map, `mapped`): only one of the two is read.
int32_t attention_impl(const char* name, bool mapped, const void* q, const void* k,
                       const void* v, const int32_t* cand_offsets, const int32_t* cand_ids,
                       const int32_t* kv_offsets, int64_t R, int64_t N, int32_t q_len,
                       int32_t num_heads, int32_t head_dim, int64_t kv_row_stride,
                       float softmax_scale, int32_t dtype, void* out, void* stream,
                       void* workspace = nullptr, size_t workspace_bytes = 0,
                       const void* residual = nullptr, void* out_sum = nullptr,
                       const void* proj_w = nullptr, int64_t proj_in = 0,
                       const void* plan = nullptr, size_t plan_bytes = 0) {
  if (!valid_dtype(dtype)) return fail(ROCS_ERR_INVALID_ARGUMENT, "unknown dtype %d", dtype);
  if (R < 0 || N < 0 || q_len < 1 || num_heads < 1 || head_dim < 1 || kv_row_stride < 0)
    return fail(ROCS_ERR_INVALID_ARGUMENT,
                "need R >= 0, N >= 0, q_len >= 1, num_heads >= 1, head_dim >= 1, "
                "kv_row_stride >= 0");
  if (head_dim > 256) return fail(ROCS_ERR_UNSUPPORTED, "head_dim %d > 256", head_dim);
  const int64_t row_elems = (int64_t)num_heads * head_dim;
  const int64_t stride = kv_row_stride == 0 ? row_elems : kv_row_stride;
  if (stride < row_elems)
    return fail(ROCS_ERR_INVALID_ARGUMENT, "kv_row_stride %lld < num_heads * head_dim",
                (long long)kv_row_stride);
  if (N * q_len > kMaxI32 || R > kMaxI32 || (int64_t)num_heads > 65535)
    return fail(ROCS_ERR_UNSUPPORTED, "batch too large");
  if (N == 0) return ok();
  if (R == 0) return fail(ROCS_ERR_INVALID_ARGUMENT, "N > 0 candidates but no requests");
  if (q == nullptr || k == nullptr || v == nullptr || out == nullptr || kv_offsets == nullptr ||
      (mapped ? cand_ids == nullptr : cand_offsets == nullptr))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "null pointer argument");
  if ((residual == nullptr) != (out_sum == nullptr))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "%s: residual and out_sum go together", name);
  if (proj_w != nullptr && (proj_in < 1 || proj_in > kMaxI32))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "%s: need 1 <= d_in < 2^31", name);
  const size_t es = esize(dtype);
  const size_t out_bytes = (size_t)N * q_len * row_elems * es;
  const size_t q_bytes = proj_w != nullptr ? (size_t)N * q_len * (size_t)proj_in * es : out_bytes;
  if (proj_w != nullptr && (overlap(out, out_bytes, proj_w, (size_t)row_elems * proj_in * es) ||
                            overlap(out_sum, out_bytes, proj_w, (size_t)row_elems * proj_in * es) ||
                            overlap(out_sum, out_bytes, q, q_bytes)))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "%s: an output overlaps x or w_q", name);
  if (overlap(out, out_bytes, q, q_bytes) || overlap(out, out_bytes, k, 1) ||
      overlap(out, out_bytes, v, 1) ||
      overlap(out, out_bytes, cand_offsets, (size_t)(R + 1) * 4) ||
      overlap(out, out_bytes, cand_ids, (size_t)N * 4) ||
      overlap(out, out_bytes, kv_offsets, (size_t)(R + 1) * 4))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "out overlaps an input");
  if (out_sum != nullptr &&
      (overlap(out_sum, out_bytes, q, out_bytes) || overlap(out_sum, out_bytes, k, 1) ||
       overlap(out_sum, out_bytes, v, 1) || overlap(out_sum, out_bytes, out, out_bytes) ||
       overlap(out_sum, out_bytes, residual, out_bytes) ||
       overlap(out_sum, out_bytes, cand_offsets, (size_t)(R + 1) * 4) ||
       overlap(out_sum, out_bytes, kv_offsets, (size_t)(R + 1) * 4) ||
       overlap(out, out_bytes, residual, out_bytes)))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "%s: out_sum overlaps an input or out, or out "
                "overlaps residual", name);
  if (plan != nullptr) {
    if (plan_bytes < rocs::attention_plan_bytes(R))
      return fail(ROCS_ERR_WORKSPACE_TOO_SMALL, "%s: plan needs %zu bytes, got %zu", name,
                  rocs::attention_plan_bytes(R), plan_bytes);
    if (!aligned(plan, 4) || overlap(out, out_bytes, plan, plan_bytes) ||
        overlap(out_sum, out_bytes, plan, plan_bytes))
      return fail(ROCS_ERR_INVALID_ARGUMENT, "%s: plan misaligned or overlapping an output",
                  name);
  }

  rocs::AttentionArgs a{};
  a.q = q; a.k = k; a.v = v; a.cand_offsets = cand_offsets; a.kv_offsets = kv_offsets;
  a.R = R; a.N = N; a.q_len = q_len; a.heads = num_heads; a.head_dim = head_dim;
  a.kv_stride = stride;
  a.scale = softmax_scale > 0.f ? softmax_scale : 1.0f / sqrtf((float)head_dim);
  a.bf16 = dtype == ROCS_DTYPE_BF16;
  a.out = out;
  a.ids = mapped ? cand_ids : nullptr;
  a.residual = residual;
  a.out_sum = out_sum;
  a.proj_w = proj_w;
  a.proj_in = (int)proj_in;
  a.plan = static_cast<const int32_t*>(plan);
  const bool fast = a.bf16 && (head_dim == 64 || head_dim == 128) && stride % 8 == 0 &&
                    stride < (int64_t(1) << 24) &&
                    aligned(q, 16) && aligned(k, 16) && aligned(v, 16) && aligned(out, 16) &&
                    aligned(residual, 16) && aligned(out_sum, 16) && aligned(proj_w, 16);
  // Launch limits: a grid may hold fewer than 2^32 work items. The general
  // kernel runs one 64-lane wave per (query row, head) with the rows on the
  // grid's x axis; the tiled kernel runs 256 lanes per (head, tile slot),
  // R + ceil(N q_len / 128) slots per head.
  // The mapped form runs the tiled kernel on the candidates grouped by
  // request when the grouping fits (R and the per-block count table), with
  // the grouping in the caller's workspace; otherwise the general kernel.
  const size_t group_bytes = mapped ? rocs::mapped_grouping_bytes(R, N) : 0;
  const bool tiled = fast && (!mapped || group_bytes > 0);
  if (mapped && tiled) {
    if (workspace == nullptr || workspace_bytes < group_bytes)
      return fail(ROCS_ERR_WORKSPACE_TOO_SMALL, "%s: workspace needs %zu bytes, got %zu", name,
                  group_bytes, workspace == nullptr ? (size_t)0 : workspace_bytes);
    if (!aligned(workspace, 256))
      return fail(ROCS_ERR_INVALID_ARGUMENT, "%s: workspace must be 256-byte aligned", name);
    if (overlap(workspace, group_bytes, out, out_bytes) ||
        overlap(workspace, group_bytes, q, out_bytes) ||
        overlap(workspace, group_bytes, cand_ids, (size_t)N * 4) ||
        overlap(workspace, group_bytes, kv_offsets, (size_t)(R + 1) * 4))
      return fail(ROCS_ERR_INVALID_ARGUMENT, "%s: workspace overlaps an argument", name);
  }
  if (!tiled && (N * q_len) >= (int64_t(1) << 26))
    return fail(ROCS_ERR_UNSUPPORTED, "%s: N * q_len = %lld query rows exceed the general "
                "kernel's grid (2^26 rows)", name, (long long)(N * q_len));
  if (tiled && (R + (N * q_len + 127) / 128) * num_heads >= (int64_t(1) << 24))
    return fail(ROCS_ERR_UNSUPPORTED, "%s: (R + N * q_len / 128) * num_heads tiles exceed the "
                "grid limit (2^24)", name);
  a.workspace = mapped && tiled ? workspace : nullptr;
  const hipError_t e = rocs::launch_attention(a, fast, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return launch_failed(name, e);
  return ok();
}

}  // namespace

extern "C" {

int32_t rocs_dca_attention(const void* q, const void* k, const void* v,
                           const int32_t* cand_offsets, const int32_t* kv_offsets, int64_t R,
                           int64_t N, int32_t q_len, int32_t num_heads, int32_t head_dim,
                           int64_t kv_row_stride, float softmax_scale, int32_t dtype, void* out,
                           void* stream) {
  return attention_impl("rocs_dca_attention", false, q, k, v, cand_offsets, nullptr,
                        kv_offsets, R, N, q_len, num_heads, head_dim, kv_row_stride,
                        softmax_scale, dtype, out, stream);
}

int32_t rocs_dca_attention_residual(const void* q, const void* k, const void* v,
                                    const int32_t* cand_offsets, const int32_t* kv_offsets,
                                    int64_t R, int64_t N, int32_t q_len, int32_t num_heads,
                                    int32_t head_dim, int64_t kv_row_stride,
                                    float softmax_scale, int32_t dtype, const void* residual,
                                    void* out, void* out_sum, void* stream) {
  if (residual == nullptr || out_sum == nullptr)
    return fail(ROCS_ERR_INVALID_ARGUMENT, "rocs_dca_attention_residual: null residual or out_sum");
  return attention_impl("rocs_dca_attention_residual", false, q, k, v, cand_offsets, nullptr,
                        kv_offsets, R, N, q_len, num_heads, head_dim, kv_row_stride,
                        softmax_scale, dtype, out, stream, nullptr, 0, residual, out_sum);
}

int32_t rocs_dca_attention_ex(const void* q, int64_t d_in, const void* w_q, const void* k,
                              const void* v, const int32_t* cand_offsets,
                              const int32_t* kv_offsets, const void* plan, size_t plan_bytes,
                              int64_t R, int64_t N, int32_t q_len, int32_t num_heads,
                              int32_t head_dim, int64_t kv_row_stride, float softmax_scale,
                              int32_t dtype, const void* residual, void* out, void* out_sum,
                              void* stream) {
  return attention_impl("rocs_dca_attention_ex", false, q, k, v, cand_offsets, nullptr,
                        kv_offsets, R, N, q_len, num_heads, head_dim, kv_row_stride,
                        softmax_scale, dtype, out, stream, nullptr, 0, residual, out_sum, w_q,
                        w_q != nullptr ? d_in : 0, plan, plan_bytes);
}

size_t rocs_dca_attention_plan_size(int64_t num_requests) {
  if (num_requests < 0 || num_requests > kMaxI32) return 0;
  return rocs::attention_plan_bytes(num_requests);
}

int32_t rocs_dca_attention_plan(const int32_t* cand_offsets, const int32_t* kv_offsets,
                                int64_t R, int64_t N, int32_t q_len, int32_t num_heads,
                                void* plan, size_t plan_bytes, void* stream) {
  static const char* name = "rocs_dca_attention_plan";
  if (R < 0 || N < 0 || q_len < 1 || num_heads < 1)
    return fail(ROCS_ERR_INVALID_ARGUMENT, "%s: need R >= 0, N >= 0, q_len >= 1, "
                "num_heads >= 1", name);
  if (R > kMaxI32 || N * q_len > kMaxI32 || num_heads > 65535 ||
      (R + (N * q_len + 127) / 128) * num_heads >= (int64_t(1) << 24))
    return fail(ROCS_ERR_UNSUPPORTED, "%s: (R + N * q_len / 128) * num_heads tiles exceed the "
                "tiled kernel's grid limit (2^24)", name);
  if (plan == nullptr || (R > 0 && (cand_offsets == nullptr || kv_offsets == nullptr)))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "%s: null pointer argument", name);
  if (plan_bytes < rocs::attention_plan_bytes(R))
    return fail(ROCS_ERR_WORKSPACE_TOO_SMALL, "%s: plan needs %zu bytes, got %zu", name,
                rocs::attention_plan_bytes(R), plan_bytes);
  if (!aligned(plan, 4))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "%s: plan must be 4-byte aligned", name);
  if (overlap(plan, plan_bytes, cand_offsets, (size_t)(R + 1) * 4) ||
      overlap(plan, plan_bytes, kv_offsets, (size_t)(R + 1) * 4))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "%s: plan overlaps the offsets", name);
  const hipError_t e = rocs::launch_attention_plan(cand_offsets, kv_offsets, R, q_len,
                                                   num_heads, static_cast<int32_t*>(plan),
                                                   static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return launch_failed(name, e);
  return ok();
}

size_t rocs_dca_attention_mapped_workspace_size(int64_t num_requests, int64_t num_cand) {
  if (num_requests <= 0 || num_cand <= 0) return 0;
  return rocs::mapped_grouping_bytes(num_requests, num_cand);
}

int32_t rocs_dca_attention_mapped(const void* q, const void* k, const void* v,
                                  const int32_t* cand_request_ids, const int32_t* kv_offsets,
                                  int64_t R, int64_t N, int32_t q_len, int32_t num_heads,
                                  int32_t head_dim, int64_t kv_row_stride, float softmax_scale,
                                  int32_t dtype, void* out, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  return attention_impl("rocs_dca_attention_mapped", true, q, k, v, nullptr, cand_request_ids,
                        kv_offsets, R, N, q_len, num_heads, head_dim, kv_row_stride,
                        softmax_scale, dtype, out, stream, workspace, workspace_bytes);
}

int32_t rocs_glm_interaction(const void* x_req, const void* x_cand, const int32_t* cand_offsets,
                             int64_t R, int64_t N, int32_t f_req, int32_t f_cand, int32_t emb,
                             int32_t dtype, void* y_req, void* y_cand, void* stream) {
  if (!valid_dtype(dtype)) return fail(ROCS_ERR_INVALID_ARGUMENT, "unknown dtype %d", dtype);
  if (R < 0 || N < 0 || f_req < 1 || f_cand < 1 || emb < 1)
    return fail(ROCS_ERR_INVALID_ARGUMENT,
                "need R >= 0, N >= 0, f_req >= 1, f_cand >= 1, emb_dim >= 1");
  if (R > kMaxI32 || N * f_cand > kMaxI32)
    return fail(ROCS_ERR_UNSUPPORTED, "batch too large");
  if (N > 0 && R == 0) return fail(ROCS_ERR_INVALID_ARGUMENT, "N > 0 candidates but no requests");
  if (y_cand == nullptr) N = 0;
  if (R == 0 || (N == 0 && y_req == nullptr)) return ok();
  if (x_req == nullptr || (N > 0 && (x_cand == nullptr || cand_offsets == nullptr)))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "null pointer argument");
  if (cand_offsets == nullptr)
    return fail(ROCS_ERR_INVALID_ARGUMENT, "cand_offsets must not be NULL");
  const size_t es = esize(dtype);
  const size_t yr_bytes = (size_t)R * f_req * f_req * es;
  const size_t yc_bytes = (size_t)N * f_cand * (f_req + f_cand) * es;
  const size_t xr_bytes = (size_t)R * f_req * emb * es, xc_bytes = (size_t)N * f_cand * emb * es;
  if (overlap(y_req, yr_bytes, x_req, xr_bytes) || overlap(y_req, yr_bytes, x_cand, xc_bytes) ||
      overlap(y_cand, yc_bytes, x_req, xr_bytes) || overlap(y_cand, yc_bytes, x_cand, xc_bytes) ||
      overlap(y_req, yr_bytes, y_cand, yc_bytes))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "outputs overlap inputs or each other");

  rocs::InteractionArgs a{};
  a.x_req = x_req; a.x_cand = x_cand; a.cand_offsets = cand_offsets;
  a.R = R; a.N = N; a.f_req = f_req; a.f_cand = f_cand; a.emb = emb;
  a.bf16 = dtype == ROCS_DTYPE_BF16;
  a.y_req = y_req; a.y_cand = N > 0 ? y_cand : nullptr;
  const bool fast = a.bf16 && f_req % 16 == 0 && (f_cand == 4 || f_cand == 8 || f_cand == 16) &&
                    emb % 32 == 0 && aligned(x_req, 16) && aligned(x_cand, 16) &&
                    aligned(y_req, 16) && aligned(y_cand, 16);
  const hipError_t e = rocs::launch_interaction(a, fast, static_cast<hipStream_t>(stream));
  if (e != hipSuccess)
    return launch_failed("rocs_glm_interaction", e);
  return ok();
}

size_t rocs_ikbo_lcb_workspace_size(int64_t num_requests, int64_t o_cand, int64_t emb_dim) {
  if (num_requests <= 0 || o_cand <= 0 || emb_dim <= 0) return 0;
  return align256((size_t)num_requests * (size_t)o_cand * (size_t)emb_dim * sizeof(float));
}

}  // extern "C"

namespace {

int32_t lcb_impl(const char* name, bool mapped, const void* x_req, const void* x_cand,
                 const void* w_rr, const void* w_cr, const void* w_cc,
                 const int32_t* cand_offsets, const int32_t* cand_ids, int64_t R, int64_t N,
                 int32_t f_req, int32_t f_cand, int32_t o_req, int32_t o_cand, int32_t emb,
                 int32_t dtype, void* y_req, void* y_cand, void* workspace,
                 size_t workspace_bytes, void* stream) {
  if (!valid_dtype(dtype)) return fail(ROCS_ERR_INVALID_ARGUMENT, "unknown dtype %d", dtype);
  if (R < 0 || N < 0 || f_req < 1 || f_cand < 1 || o_req < 0 || o_cand < 1 || emb < 1)
    return fail(ROCS_ERR_INVALID_ARGUMENT,
                "need R >= 0, N >= 0, f_req >= 1, f_cand >= 1, o_req >= 0, o_cand >= 1, "
                "emb_dim >= 1");
  if (R > kMaxI32 || N > kMaxI32 || (int64_t)f_cand * emb > (1 << 24) ||
      (int64_t)f_req * emb > (1 << 24) || (int64_t)(o_req + o_cand) * emb > (1 << 24))
    return fail(ROCS_ERR_UNSUPPORTED, "size too large");
  if (y_req == nullptr) o_req = 0;
  // One thread per output element in the request kernel (and the general
  // candidate kernel): keep both grids below 2^31 workgroups.
  if (R * (int64_t)(o_req + o_cand) * emb / 256 >= kMaxI32 ||
      N * (int64_t)o_cand * emb / 256 >= kMaxI32)
    return fail(ROCS_ERR_UNSUPPORTED, "batch too large");
  if (R == 0) {
    if (N > 0) return fail(ROCS_ERR_INVALID_ARGUMENT, "N > 0 candidates but no requests");
    return ok();
  }
  if (x_req == nullptr || w_cr == nullptr || (o_req > 0 && w_rr == nullptr) ||
      (N > 0 && (x_cand == nullptr || w_cc == nullptr || y_cand == nullptr ||
                 (mapped ? cand_ids == nullptr : cand_offsets == nullptr))))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "null pointer argument");
  const size_t need = rocs_ikbo_lcb_workspace_size(R, o_cand, emb);
  if (workspace == nullptr || workspace_bytes < need)
    return fail(ROCS_ERR_WORKSPACE_TOO_SMALL, "workspace needs %zu bytes, got %zu", need,
                workspace == nullptr ? (size_t)0 : workspace_bytes);
  if (!aligned(workspace, 256))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  const size_t es = esize(dtype);
  const size_t yr_bytes = (size_t)R * o_req * emb * es, yc_bytes = (size_t)N * o_cand * emb * es;
  const struct { const void* p; size_t n; } ins[] = {
      {x_req, (size_t)R * f_req * emb * es}, {x_cand, (size_t)N * f_cand * emb * es},
      {w_rr, (size_t)o_req * f_req * es}, {w_cr, (size_t)o_cand * f_req * es},
      {w_cc, (size_t)o_cand * f_cand * es}, {cand_offsets, (size_t)(R + 1) * 4},
      {cand_ids, (size_t)N * 4}};
  for (const auto& in : ins)
    if (overlap(y_req, yr_bytes, in.p, in.n) || overlap(y_cand, yc_bytes, in.p, in.n) ||
        overlap(workspace, need, in.p, in.n))
      return fail(ROCS_ERR_INVALID_ARGUMENT, "an output or the workspace overlaps an input");
  if (overlap(y_req, yr_bytes, y_cand, yc_bytes) || overlap(y_req, yr_bytes, workspace, need) ||
      overlap(y_cand, yc_bytes, workspace, need))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "outputs and workspace overlap");

  rocs::LcbArgs a{};
  a.x_req = x_req; a.x_cand = x_cand; a.w_rr = w_rr; a.w_cr = w_cr; a.w_cc = w_cc;
  a.cand_offsets = mapped ? nullptr : cand_offsets;
  a.ids = mapped ? cand_ids : nullptr;
  a.R = R; a.N = N; a.f_req = f_req; a.f_cand = f_cand; a.o_req = o_req; a.o_cand = o_cand;
  a.emb = emb; a.bf16 = dtype == ROCS_DTYPE_BF16;
  a.y_req = o_req > 0 ? y_req : nullptr; a.y_cand = y_cand;
  a.z = static_cast<float*>(workspace);
  const bool fast = a.bf16 && rocs::lcb_fast_shape(f_cand, o_cand, emb) && aligned(x_cand, 16) &&
                    aligned(w_cc, 8) && aligned(y_cand, 16) && aligned(x_req, 8) &&
                    aligned(y_req, 8);
  const hipError_t e = rocs::launch_lcb(a, fast, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return launch_failed(name, e);
  return ok();
}

}  // namespace

extern "C" {

int32_t rocs_ikbo_lcb(const void* x_req, const void* x_cand, const void* w_rr, const void* w_cr,
                      const void* w_cc, const int32_t* cand_offsets, int64_t R, int64_t N,
                      int32_t f_req, int32_t f_cand, int32_t o_req, int32_t o_cand,
                      int32_t emb_dim, int32_t dtype, void* y_req, void* y_cand,
                      void* workspace, size_t workspace_bytes, void* stream) {
  return lcb_impl("rocs_ikbo_lcb", false, x_req, x_cand, w_rr, w_cr, w_cc, cand_offsets,
                  nullptr, R, N, f_req, f_cand, o_req, o_cand, emb_dim, dtype, y_req, y_cand,
                  workspace, workspace_bytes, stream);
}

int32_t rocs_ikbo_lcb_mapped(const void* x_req, const void* x_cand, const void* w_rr,
                             const void* w_cr, const void* w_cc,
                             const int32_t* cand_request_ids, int64_t R, int64_t N,
                             int32_t f_req, int32_t f_cand, int32_t o_req, int32_t o_cand,
                             int32_t emb_dim, int32_t dtype, void* y_req, void* y_cand,
                             void* workspace, size_t workspace_bytes, void* stream) {
  return lcb_impl("rocs_ikbo_lcb_mapped", true, x_req, x_cand, w_rr, w_cr, w_cc, nullptr,
                  cand_request_ids, R, N, f_req, f_cand, o_req, o_cand, emb_dim, dtype, y_req,
                  y_cand, workspace, workspace_bytes, stream);
}

// The fused two-layer kernel's shapes (bf16). Other shapes and fp32 run the
// two-launch form, which keeps H in the workspace.
static bool mlp2_fused(int64_t R, int64_t k_req, int64_t k_cand, int64_t d_hidden,
                       int64_t d_out, int32_t dtype) {
  return dtype == ROCS_DTYPE_BF16 && k_req % 8 == 0 &&
         rocs::mlp2_fused_shape(R, k_cand, d_hidden, d_out);
}

size_t rocs_ikbo_mlp2_workspace_size(int64_t num_requests, int64_t num_cand, int64_t k_req,
                                     int64_t k_cand, int64_t d_hidden, int64_t d_out,
                                     int32_t dtype) {
  if (num_requests < 0 || num_cand <= 0 || k_req < 0 || k_cand < 1 || d_hidden < 1 ||
      d_out < 1 || !valid_dtype(dtype))
    return 0;
  size_t n = 0;
  const bool req = k_req > 0 && num_requests > 0;
  // Request table Zb [R, d_hidden] fp32.
  if (req) n += align256((size_t)num_requests * (size_t)d_hidden * sizeof(float));
  if (!mlp2_fused(num_requests, k_req, k_cand, d_hidden, d_out, dtype)) {
    if (req) n += align256((size_t)num_cand * sizeof(int32_t));   // index map
    n += align256((size_t)num_cand * (size_t)d_hidden * esize(dtype));   // H
  }
  return n;
}

int32_t rocs_ikbo_mlp2(const void* x_req, int64_t k_req, const void* x_cand, int64_t k_cand,
                       const void* w1_req, const void* w1_cand, const float* b1,
                       const void* w2, const float* b2, const int32_t* cand_offsets,
                       int64_t R, int64_t N, int64_t d_hidden, int64_t d_out, int32_t dtype,
                       int32_t activation1, int32_t activation2, void* out, void* workspace,
                       size_t workspace_bytes, void* stream) {
  if (!valid_dtype(dtype)) return fail(ROCS_ERR_INVALID_ARGUMENT, "unknown dtype %d", dtype);
  for (int32_t act : {activation1, activation2})
    if (act != ROCS_ACT_NONE && act != ROCS_ACT_RELU)
      return fail(ROCS_ERR_INVALID_ARGUMENT, "unknown activation %d", act);
  if (R < 0 || N < 0 || k_req < 0 || k_cand < 1 || d_hidden < 1 || d_out < 1)
    return fail(ROCS_ERR_INVALID_ARGUMENT,
                "sizes must satisfy R >= 0, N >= 0, k_req >= 0, k_cand >= 1, d_hidden >= 1, "
                "d_out >= 1");
  if (R > kMaxI32 || N > kMaxI32 || k_req > kMaxI32 || k_cand > kMaxI32 ||
      d_hidden > kMaxI32 || d_out > kMaxI32)
    return fail(ROCS_ERR_UNSUPPORTED, "a size exceeds 2^31 - 1");
  if (N == 0) return ok();
  if (k_req > 0 && R == 0)
    return fail(ROCS_ERR_INVALID_ARGUMENT, "N > 0 candidates but no requests to own them");
  if (x_cand == nullptr || w1_cand == nullptr || w2 == nullptr || out == nullptr)
    return fail(ROCS_ERR_INVALID_ARGUMENT, "x_cand, w1_cand, w2 and out must not be NULL");
  if (k_req > 0 && (x_req == nullptr || w1_req == nullptr || cand_offsets == nullptr))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "k_req > 0 needs x_req, w1_req and cand_offsets");
  const bool fused = mlp2_fused(R, k_req, k_cand, d_hidden, d_out, dtype);
  if (fused && !(aligned(x_cand, 16) && aligned(w1_cand, 16) && aligned(w2, 16) &&
                 aligned(out, 16) && aligned(b1, 16) && aligned(b2, 16) &&
                 aligned(x_req, 16) && aligned(w1_req, 16)))
    return fail(ROCS_ERR_INVALID_ARGUMENT,
                "the fused kernel needs 16-byte aligned x_req, x_cand, w1_req, w1_cand, b1, "
                "w2, b2 and out");
  const size_t need = rocs_ikbo_mlp2_workspace_size(R, N, k_req, k_cand, d_hidden, d_out, dtype);
  if (need > 0) {
    if (workspace == nullptr || workspace_bytes < need)
      return fail(ROCS_ERR_WORKSPACE_TOO_SMALL, "workspace needs %zu bytes, got %zu", need,
                  workspace == nullptr ? (size_t)0 : workspace_bytes);
    if (!aligned(workspace, 256))
      return fail(ROCS_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  }
  const size_t es = esize(dtype);
  const size_t out_bytes = (size_t)N * d_out * es;
  const struct { const void* p; size_t n; const char* name; } ins[] = {
      {x_req, (size_t)R * k_req * es, "x_req"},
      {x_cand, (size_t)N * k_cand * es, "x_cand"},
      {w1_req, (size_t)d_hidden * k_req * es, "w1_req"},
      {w1_cand, (size_t)d_hidden * k_cand * es, "w1_cand"},
      {b1, (size_t)d_hidden * sizeof(float), "b1"},
      {w2, (size_t)d_out * d_hidden * es, "w2"},
      {b2, (size_t)d_out * sizeof(float), "b2"},
      {cand_offsets, (size_t)(R + 1) * sizeof(int32_t), "cand_offsets"},
  };
  for (const auto& in : ins) {
    if (overlap(out, out_bytes, in.p, in.n))
      return fail(ROCS_ERR_INVALID_ARGUMENT, "out overlaps %s", in.name);
    if (need > 0 && overlap(workspace, need, in.p, in.n))
      return fail(ROCS_ERR_INVALID_ARGUMENT, "workspace overlaps %s", in.name);
  }
  if (need > 0 && overlap(workspace, need, out, out_bytes))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "workspace overlaps out");
  // One workgroup per 128-candidate tile slot.
  if (R + N / 128 + 1 >= kMaxI32) return fail(ROCS_ERR_UNSUPPORTED, "batch too large");

  rocs::Mlp2Args a{};
  a.x_req = x_req; a.x_cand = x_cand; a.cand_offsets = cand_offsets;
  a.w1_req = w1_req; a.w1_cand = w1_cand; a.b1 = b1; a.w2 = w2; a.b2 = b2;
  a.R = R; a.N = N; a.k_req = k_req; a.k_cand = k_cand; a.d_hidden = d_hidden; a.d_out = d_out;
  a.bf16 = dtype == ROCS_DTYPE_BF16;
  a.relu1 = activation1 == ROCS_ACT_RELU;
  a.relu2 = activation2 == ROCS_ACT_RELU;
  a.out = out;
  char* ws = static_cast<char*>(workspace);
  size_t at = 0;
  if (k_req > 0) {
    a.z = reinterpret_cast<float*>(ws);
    at = align256((size_t)R * d_hidden * sizeof(float));
  }
  if (!fused) {
    if (k_req > 0) {
      a.ids = reinterpret_cast<int32_t*>(ws + at);
      at += align256((size_t)N * sizeof(int32_t));
    }
    a.h = ws + at;
    a.linear_fast = a.bf16 && k_cand % 8 == 0 && k_req % 8 == 0 && d_hidden % 8 == 0 &&
                    d_out % 4 == 0 && aligned(x_cand, 16) && aligned(w1_cand, 16) &&
                    aligned(x_req, 16) && aligned(w1_req, 16) && aligned(b1, 16) &&
                    aligned(w2, 16) && aligned(b2, 16) && aligned(out, 16);
  }
  const hipError_t e = rocs::launch_mlp2(a, fused, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return launch_failed("rocs_ikbo_mlp2", e);
  return ok();
}

static bool fm_linear_fused(int32_t f_req, int32_t f_cand, int32_t emb, int64_t d_out,
                            int32_t dtype) {
  return dtype == ROCS_DTYPE_BF16 && rocs::fm_linear_fused_shape(f_req, f_cand, emb, d_out);
}

size_t rocs_glm_fm_linear_workspace_size(int64_t num_requests, int64_t num_cand, int32_t f_req,
                                         int32_t f_cand, int32_t emb_dim, int64_t d_out,
                                         int32_t dtype) {
  if (num_requests <= 0 || num_cand < 0 || f_req < 1 || f_cand < 1 || emb_dim < 1 ||
      d_out < 1 || !valid_dtype(dtype))
    return 0;
  const size_t es = esize(dtype);
  // Y^R [R, f_req^2], then Zb [R, d_out] fp32.
  size_t n = align256((size_t)num_requests * f_req * f_req * es) +
             align256((size_t)num_requests * (size_t)d_out * sizeof(float));
  if (!fm_linear_fused(f_req, f_cand, emb_dim, d_out, dtype))   // Y^C and the index map
    n += align256((size_t)num_cand * f_cand * (f_req + f_cand) * es) +
         align256((size_t)num_cand * sizeof(int32_t));
  return n;
}

int32_t rocs_glm_fm_linear(const void* x_req, const void* x_cand, const int32_t* cand_offsets,
                           int64_t R, int64_t N, int32_t f_req, int32_t f_cand, int32_t emb,
                           const void* w_req, const void* w_cand, const float* bias,
                           int64_t d_out, int32_t dtype, int32_t activation, void* out,
                           void* workspace, size_t workspace_bytes, void* stream) {
  if (!valid_dtype(dtype)) return fail(ROCS_ERR_INVALID_ARGUMENT, "unknown dtype %d", dtype);
  if (activation != ROCS_ACT_NONE && activation != ROCS_ACT_RELU)
    return fail(ROCS_ERR_INVALID_ARGUMENT, "unknown activation %d", activation);
  if (R < 0 || N < 0 || f_req < 1 || f_cand < 1 || emb < 1 || d_out < 1)
    return fail(ROCS_ERR_INVALID_ARGUMENT,
                "need R >= 0, N >= 0, f_req >= 1, f_cand >= 1, emb_dim >= 1, d_out >= 1");
  const int64_t k_req = (int64_t)f_req * f_req, k_cand = (int64_t)f_cand * (f_req + f_cand);
  if (R > kMaxI32 || N * f_cand > kMaxI32 || N * k_cand > kMaxI32 || R * k_req > kMaxI32 ||
      d_out > kMaxI32 || (int64_t)f_req * emb > (1 << 24) || (int64_t)f_cand * emb > (1 << 24))
    return fail(ROCS_ERR_UNSUPPORTED, "size too large");
  if (N == 0) return ok();
  if (R == 0) return fail(ROCS_ERR_INVALID_ARGUMENT, "N > 0 candidates but no requests");
  if (x_req == nullptr || x_cand == nullptr || cand_offsets == nullptr || w_req == nullptr ||
      w_cand == nullptr || out == nullptr)
    return fail(ROCS_ERR_INVALID_ARGUMENT, "null pointer argument");
  const bool fused = fm_linear_fused(f_req, f_cand, emb, d_out, dtype);
  if (fused && !(aligned(x_req, 16) && aligned(x_cand, 16) && aligned(w_req, 16) &&
                 aligned(w_cand, 16) && aligned(bias, 16) && aligned(out, 16)))
    return fail(ROCS_ERR_INVALID_ARGUMENT,
                "the fused kernel needs 16-byte aligned x_req, x_cand, w_req, w_cand, bias "
                "and out");
  const size_t need = rocs_glm_fm_linear_workspace_size(R, N, f_req, f_cand, emb, d_out, dtype);
  if (workspace == nullptr || workspace_bytes < need)
    return fail(ROCS_ERR_WORKSPACE_TOO_SMALL, "workspace needs %zu bytes, got %zu", need,
                workspace == nullptr ? (size_t)0 : workspace_bytes);
  if (!aligned(workspace, 256))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  const size_t es = esize(dtype);
  const size_t out_bytes = (size_t)N * d_out * es;
  const struct { const void* p; size_t n; const char* name; } ins[] = {
      {x_req, (size_t)R * f_req * emb * es, "x_req"},
      {x_cand, (size_t)N * f_cand * emb * es, "x_cand"},
      {cand_offsets, (size_t)(R + 1) * sizeof(int32_t), "cand_offsets"},
      {w_req, (size_t)d_out * k_req * es, "w_req"},
      {w_cand, (size_t)d_out * k_cand * es, "w_cand"},
      {bias, (size_t)d_out * sizeof(float), "bias"},
  };
  for (const auto& in : ins) {
    if (overlap(out, out_bytes, in.p, in.n))
      return fail(ROCS_ERR_INVALID_ARGUMENT, "out overlaps %s", in.name);
    if (overlap(workspace, need, in.p, in.n))
      return fail(ROCS_ERR_INVALID_ARGUMENT, "workspace overlaps %s", in.name);
  }
  if (overlap(workspace, need, out, out_bytes))
    return fail(ROCS_ERR_INVALID_ARGUMENT, "workspace overlaps out");

  rocs::FmLinearArgs a{};
  a.x_req = x_req; a.x_cand = x_cand; a.cand_offsets = cand_offsets;
  a.w_req = w_req; a.w_cand = w_cand; a.bias = bias;
  a.R = R; a.N = N; a.d_out = d_out; a.f_req = f_req; a.f_cand = f_cand; a.emb = emb;
  a.bf16 = dtype == ROCS_DTYPE_BF16;
  a.relu = activation == ROCS_ACT_RELU;
  a.out = out;
  char* ws = static_cast<char*>(workspace);
  a.y_req = ws;
  size_t at = align256((size_t)R * k_req * es);
  a.z = reinterpret_cast<float*>(ws + at);
  at += align256((size_t)R * d_out * sizeof(float));
  if (!fused) {
    a.y_cand = ws + at;
    at += align256((size_t)N * k_cand * es);
    a.ids = reinterpret_cast<int32_t*>(ws + at);
  }
  a.interaction_fast = a.bf16 && f_req % 16 == 0 &&
                       (f_cand == 4 || f_cand == 8 || f_cand == 16) && emb % 32 == 0 &&
                       aligned(x_req, 16) && aligned(x_cand, 16);
  a.linear_fast = a.bf16 && k_cand % 8 == 0 && k_req % 8 == 0 && d_out % 4 == 0 &&
                  aligned(w_req, 16) && aligned(w_cand, 16) && aligned(bias, 16) &&
                  aligned(out, 16);
  const hipError_t e = rocs::launch_fm_linear(a, fused, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return launch_failed("rocs_glm_fm_linear", e);
  return ok();
}

int32_t rocs_request_ids(const int32_t* cand_offsets, int64_t R, int64_t N, int32_t* out_ids,
                         void* stream) {
  if (R < 0 || N < 0) return fail(ROCS_ERR_INVALID_ARGUMENT, "negative size");
  if (N > kMaxI32 || R > kMaxI32) return fail(ROCS_ERR_UNSUPPORTED, "batch too large");
  if (N == 0) return ok();
  if (R == 0) return fail(ROCS_ERR_INVALID_ARGUMENT, "N > 0 candidates but no requests");
  if (cand_offsets == nullptr || out_ids == nullptr)
    return fail(ROCS_ERR_INVALID_ARGUMENT, "null pointer argument");
  const hipError_t e = rocs::launch_request_ids(cand_offsets, R, N, out_ids,
                                                static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return launch_failed("rocs_request_ids", e);
  return ok();
}

int32_t rocs_validate_offsets(const int32_t* offsets, int64_t count, int64_t total,
                              void* stream) {
  if (offsets == nullptr || count < 1)
    return fail(ROCS_ERR_INVALID_ARGUMENT, "need a non-NULL offsets array of count >= 1");
  std::vector<int32_t> h((size_t)count);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(h.data(), offsets, (size_t)count * sizeof(int32_t),
                                hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return fail(ROCS_ERR_HIP, "rocs_validate_offsets: %s", hipGetErrorString(e));
  if (h[0] != 0) return fail(ROCS_ERR_INVALID_ARGUMENT, "offsets[0] = %d, expected 0", h[0]);
  for (int64_t i = 1; i < count; ++i)
    if (h[(size_t)i] < h[(size_t)i - 1])
      return fail(ROCS_ERR_INVALID_ARGUMENT, "offsets decrease at index %lld", (long long)i);
  if (h[(size_t)count - 1] != total)
    return fail(ROCS_ERR_INVALID_ARGUMENT, "offsets end at %d, expected %lld",
                h[(size_t)count - 1], (long long)total);
  return ok();
}

}  // extern "C"
