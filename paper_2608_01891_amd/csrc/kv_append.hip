// KV-cache append of the current decode token, gfx950.
//
// Each decode step adds the new token's key and value to the growing cache
// before attention reads it (section 1; section 2, "LLM Serving"). The new
// token is the last cached one: position j = ctx_b - 1 of sequence b.
// One thread per (sequence, kv head, 8 elements of d): the key chunk is one
// 16-byte store into the token-major K tile, the value chunk eight 2-byte
// stores into the token-fastest V tile. Sequences with ctx_b <= 0 or a
// position past the table's capacity, and out-of-range block ids, write
// nothing.
#include "common.h"
#include "kernels.h"
#include "profile.h"

namespace aflex {

__global__ __launch_bounds__(256) void kv_append_kernel(aflex_kv_append_args a) {
  const int chunks = a.D / 8;
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long long)a.B * a.Hkv * chunks) return;
  const int c = (int)(idx % chunks);
  const int h = (int)((idx / chunks) % a.Hkv);
  const int b = (int)(idx / ((long long)chunks * a.Hkv));
  const int ctx = a.context_lens[b];
  if (ctx <= 0 || ctx > a.max_blocks_per_seq * 16) return;
  const int j = ctx - 1;
  const int blk = a.block_table[(size_t)b * a.max_blocks_per_seq + j / 16];
  if (blk < 0 || blk >= a.num_blocks) return;
  const int o = j % 16;
  const size_t src = ((size_t)b * a.Hkv + h) * a.D + c * 8;
  const uint4 kv = *reinterpret_cast<const uint4*>(a.k_new + src);
  *reinterpret_cast<uint4*>(a.k_cache + (((size_t)blk * a.Hkv + h) * 16 + o) * a.D + c * 8) = kv;
  const uint4 vv = *reinterpret_cast<const uint4*>(a.v_new + src);
  const uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
  uint16_t* vdst = a.v_cache + (((size_t)blk * a.Hkv + h) * a.D + c * 8) * 16 + o;
#pragma unroll
  for (int e = 0; e < 8; ++e) vdst[e * 16] = static_cast<uint16_t>(w[e >> 1] >> ((e & 1) * 16));
}

hipError_t launch_kv_append(const aflex_kv_append_args& a, hipStream_t stream) {
  const long long n = (long long)a.B * a.Hkv * (a.D / 8);
  if (n == 0) return hipSuccess;
  ProfScope ps("kv_append", stream);
  kv_append_kernel<<<(unsigned)((n + 255) / 256), 256, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace aflex
