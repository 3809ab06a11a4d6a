// Internal launcher interface between the C ABI layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rocs {

struct LinearArgs {
  const void* x_req;
  const void* x_cand;
  const void* x_cand_add;
  const void* w_req;
  const void* w_cand;
  const float* bias;
  const int32_t* cand_offsets;
  int64_t R, N, k_req, k_cand, d_out;
  bool bf16, relu;
  void* out;
  float* z;          // [R, d_out] workspace (k_req > 0)
  int32_t* ids;      // [N] request of each candidate: workspace, or the caller's map
  bool ids_given;    // ids is the caller's map (no CSR offsets, no expansion)
  // Full GLM layer: the request-side output Y^R = act(x_req W_RR^T + b^R).
  const void* w_rr;  // [d_req, k_req]
  const float* b_rr; // [d_req] or NULL
  void* y_req;       // [R, d_req] or NULL (candidate output only)
  int64_t d_req;
  bool combined;     // run the request side inside the streaming candidate kernel
};

struct AttentionArgs {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* cand_offsets;
  const int32_t* kv_offsets;
  int64_t R, N;
  int q_len, heads, head_dim;
  int64_t kv_stride;   // elements between history rows
  float scale;
  bool bf16;
  void* out;
  const int32_t* ids;  // caller's per-candidate request map, or NULL (CSR offsets)
  void* workspace;     // grouping workspace of the mapped form (mapped_grouping_bytes), or NULL
  const void* residual;  // [N, q_len, H, d] added to the rounded output into out_sum, or NULL
  void* out_sum;
  const void* proj_w;    // W_q [H d, proj_in] when q holds X [N, q_len, proj_in], or NULL
  int proj_in;
  const int32_t* plan;   // tile order from launch_attention_plan (attention_plan_bytes(R)), or NULL
};

struct InteractionArgs {
  const void* x_req;
  const void* x_cand;
  const int32_t* cand_offsets;
  int64_t R, N;
  int f_req, f_cand, emb;
  bool bf16;
  void* y_req;
  void* y_cand;
};

struct LcbArgs {
  const void* x_req;    // [R, f_req, emb]
  const void* x_cand;   // [N, f_cand, emb]
  const void* w_rr;     // [o_req, f_req] (may be NULL when o_req == 0)
  const void* w_cr;     // [o_cand, f_req]
  const void* w_cc;     // [o_cand, f_cand]
  const int32_t* cand_offsets;   // CSR [R + 1], or NULL with ids
  const int32_t* ids;            // caller's per-candidate map, or NULL
  int64_t R, N;
  int f_req, f_cand, o_req, o_cand, emb;
  bool bf16;
  void* y_req;          // [R, o_req, emb] or NULL
  void* y_cand;         // [N, o_cand, emb]
  float* z;             // [R, o_cand, emb] workspace
};

struct Mlp2Args {
  const void* x_req;    // [R, k_req]
  const void* x_cand;   // [N, k_cand]
  const int32_t* cand_offsets;   // CSR [R + 1] (k_req > 0)
  const void* w1_req;   // [d_hidden, k_req]
  const void* w1_cand;  // [d_hidden, k_cand]
  const float* b1;      // [d_hidden] or NULL
  const void* w2;       // [d_out, d_hidden]
  const float* b2;      // [d_out] or NULL
  int64_t R, N, k_req, k_cand, d_hidden, d_out;
  bool bf16, relu1, relu2;
  bool linear_fast;     // the two-launch form may take the fast linear kernels
  void* out;            // [N, d_out]
  float* z;             // [R, d_hidden] workspace (k_req > 0)
  int32_t* ids;         // [N] workspace of the two-launch form (k_req > 0)
  void* h;              // [N, d_hidden] workspace of the two-launch form
};

struct FmLinearArgs {
  const void* x_req;    // [R, f_req, emb]
  const void* x_cand;   // [N, f_cand, emb]
  const int32_t* cand_offsets;   // CSR [R + 1]
  const void* w_req;    // [d_out, f_req^2]
  const void* w_cand;   // [d_out, f_cand (f_req + f_cand)]
  const float* bias;    // [d_out] or NULL
  int64_t R, N, d_out;
  int f_req, f_cand, emb;
  bool bf16, relu;
  bool interaction_fast, linear_fast;   // kernel choices of the two-operator form
  void* out;            // [N, d_out]
  void* y_req;          // [R, f_req^2] workspace (the request-side interaction)
  void* y_cand;         // [N, f_cand (f_req + f_cand)] workspace (two-operator form only)
  float* z;             // [R, d_out] workspace
  int32_t* ids;         // [N] workspace (two-operator form only)
};

// Each returns hipSuccess or the launch error.
hipError_t launch_request_ids(const int32_t* off, int64_t R, int64_t N, int32_t* ids,
                              hipStream_t s);
hipError_t launch_linear(const LinearArgs& a, bool fast, hipStream_t s);
hipError_t launch_attention(const AttentionArgs& a, bool fast, hipStream_t s);
// Tile order of the tiled attention kernel for one batch's offsets: longest
// history first (requests up to kAttnPlanMaxSort; beyond that the plan says
// "built-in order"). Bytes of the plan for R requests.
constexpr int64_t kAttnPlanMaxSort = 4096;
size_t attention_plan_bytes(int64_t R);
hipError_t launch_attention_plan(const int32_t* cand_off, const int32_t* kv_off, int64_t R,
                                 int q_len, int heads, int32_t* plan, hipStream_t s);
// Grouping of a per-candidate map by request for the tiled attention kernel:
// false when R or the per-block count table is too large for it (then the
// general kernel runs); the workspace it needs, 0 in that case.
bool mapped_grouping_plan(int64_t R, int64_t N, int64_t* G, int* nb);
size_t mapped_grouping_bytes(int64_t R, int64_t N);
hipError_t launch_interaction(const InteractionArgs& a, bool fast, hipStream_t s);
hipError_t launch_lcb(const LcbArgs& a, bool fast, hipStream_t s);
bool lcb_fast_shape(int f_cand, int o_cand, int emb);
// The request table Zb = x_req W_req^T + bias (fp32, [R, d_out]) alone, bf16 in.
hipError_t launch_request_table(const LinearArgs& a, hipStream_t s);
hipError_t launch_mlp2(const Mlp2Args& a, bool fused, hipStream_t s);
bool mlp2_fused_shape(int64_t R, int64_t k_cand, int64_t d_hidden, int64_t d_out);
hipError_t launch_fm_linear(const FmLinearArgs& a, bool fused, hipStream_t s);
bool fm_linear_fused_shape(int f_req, int f_cand, int emb, int64_t d_out);

}  // namespace rocs
