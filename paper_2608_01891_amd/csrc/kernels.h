// Internal launch interface between the C-ABI layer and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>

#include "aflex.h"

namespace aflex {

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Library-owned device scratch of the entry points that allocate nothing
// (scratch.hip): kStaticScratchBytes per device, shared by every such call on
// that device. static_scratch returns its device address on the current
// device (looked up once per device, then cached).
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
hipError_t static_scratch(void** ptr);

// Decode attention (attn_decode.hip). attn_shape_fits: the flattened block
// range B * Hkv * ceil(max_context_len / 16) stays below 2^30.
bool attn_shape_fits(const aflex_attn_args& a);
size_t attn_workspace_bytes(const aflex_attn_args& a);
// K/V tiles stream with non-temporal loads: every cached byte is read once,
// alone and next to the FFN's weight stream in the two-stream step alike
// (that step: 2.785 -> 2.730 ms against ordinary loads). The form of the even
// split: kAlone, three 4-wave work-groups per CU with ranges weighted by
// dispatch round (the call has the GPU to itself); kWide, one 12-wave
// work-group per CU (beside the FFN's weight stream, the pipeline step);
// kShared, three 4-wave work-groups per CU with equal ranges (beside other
// work that takes CUs first, the layer step). The workspace is the same.
enum class AttnForm { kAlone, kWide, kShared };
hipError_t launch_attn_decode(const aflex_attn_args& a, void* ws, hipStream_t stream,
                              AttnForm form = AttnForm::kAlone);

// Dense SwiGLU FFN (ffn.hip).
size_t swiglu_workspace_bytes(const aflex_ffn_args& f);
hipError_t launch_swiglu(const aflex_ffn_args& f, void* ws, hipStream_t stream);

// KV-cache append (kv_append.hip) and linear layer (ffn.hip).
hipError_t launch_kv_append(const aflex_kv_append_args& a, hipStream_t stream);
hipError_t launch_kv_write(const aflex_kv_write_args& a, hipStream_t stream);
size_t linear_workspace_bytes(const aflex_linear_args& l);
hipError_t launch_linear(const aflex_linear_args& l, void* ws, hipStream_t stream,
                         const uint16_t* residual = nullptr);

// Top-k MoE FFN (moe.hip).
size_t moe_workspace_bytes(const aflex_ffn_args& f);
// residual (optional, [T, H]) is added to the output in the combine step.
hipError_t launch_moe(const aflex_ffn_args& f, void* ws, hipStream_t stream, const uint16_t* residual = nullptr);
// The two halves of launch_moe: routing (depends only on the logits) and the
// expert computation, with separate workspace blocks.
size_t moe_route_bytes(const aflex_ffn_args& f);
size_t moe_expert_bytes(const aflex_ffn_args& f);
hipError_t launch_moe_route(const aflex_ffn_args& f, void* route_ws, hipStream_t stream);
hipError_t launch_moe_experts(const aflex_ffn_args& f, void* route_ws, void* expert_ws, hipStream_t stream,
                              const uint16_t* residual = nullptr);

// Causal prefill attention (attn_prefill.hip).
hipError_t launch_attn_prefill(const aflex_prefill_args& a, hipStream_t stream);

// RMSNorm + router + MoE block (moe_block.hip).
constexpr int kMaxRouterE = 64;
size_t moe_block_workspace_bytes(const aflex_moe_block_args& m);
hipError_t launch_moe_block(const aflex_moe_block_args& m, void* ws, hipStream_t stream);

}  // namespace aflex
