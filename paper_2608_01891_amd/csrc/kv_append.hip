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

// Packed multi-token write: one work-group per (cache block slot, sequence),
// one thread per (kv head, 8 elements of d). Slot jj of sequence b is logical
// block (max(start, 0) / 16) + jj with start = ctx_b - n_b; a thread moves the
// block's new positions: K rows as 16-byte stores, and V as whole 32-byte rows
// of the token-fastest tile when the block is entirely new (2-byte stores at a
// partial first or last block).
__global__ __launch_bounds__(1024) void kv_write_kernel(aflex_kv_write_args a) {
  const int chunks = a.D / 8;
  const int g = threadIdx.x / chunks, c = threadIdx.x % chunks;
  if (g >= a.Hkv) return;
  const int b = blockIdx.y;
  int s1 = a.cu_seqlens[b + 1], s0 = a.cu_seqlens[b];
  s1 = min(max(s1, 0), a.T);
  s0 = min(max(s0, 0), s1);
  const int n = s1 - s0, ctx = a.context_lens[b];
  if (n <= 0 || ctx <= 0 || ctx > a.max_blocks_per_seq * 16) return;
  const int start = ctx - n;
  const int jb = max(start, 0) / 16 + (int)blockIdx.x;
  const int lo = max(jb * 16, max(start, 0)), hi = min(jb * 16 + 16, ctx);
  if (lo >= hi) return;
  const int blk = a.block_table[(size_t)b * a.max_blocks_per_seq + jb];
  if (blk < 0 || blk >= a.num_blocks) return;
  const size_t row_stride = (size_t)a.Hkv * a.D;
  // new token at cache position pos is row s0 + pos - start of k_new / v_new
  const long long shift = (long long)s0 - start;
  const uint16_t* kn = a.k_new + (size_t)g * a.D + c * 8;
  const uint16_t* vn = a.v_new + (size_t)g * a.D + c * 8;
  uint16_t* kc = a.k_cache + ((size_t)blk * a.Hkv + g) * 16 * a.D + c * 8;
  uint16_t* vc = a.v_cache + (((size_t)blk * a.Hkv + g) * a.D + c * 8) * 16;
  for (int pos = lo; pos < hi; ++pos)
    *reinterpret_cast<uint4*>(kc + (size_t)(pos % 16) * a.D) =
        *reinterpret_cast<const uint4*>(kn + (size_t)(shift + pos) * row_stride);
  if (hi - lo == 16) {
    uint32_t t[16][4];
#pragma unroll
    for (int o = 0; o < 16; ++o) {
      const uint4 u = *reinterpret_cast<const uint4*>(vn + (size_t)(shift + jb * 16 + o) * row_stride);
      t[o][0] = u.x;
      t[o][1] = u.y;
      t[o][2] = u.z;
      t[o][3] = u.w;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
      uint32_t r[8];
#pragma unroll
      for (int o = 0; o < 8; ++o) r[o] = __builtin_amdgcn_perm(t[2 * o + 1][e >> 1], t[2 * o][e >> 1], sel);
      uint4* dst = reinterpret_cast<uint4*>(vc + e * 16);
      dst[0] = make_uint4(r[0], r[1], r[2], r[3]);
      dst[1] = make_uint4(r[4], r[5], r[6], r[7]);
    }
  } else {
    for (int pos = lo; pos < hi; ++pos) {
      const uint4 u = *reinterpret_cast<const uint4*>(vn + (size_t)(shift + pos) * row_stride);
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) vc[e * 16 + pos % 16] = static_cast<uint16_t>(w[e >> 1] >> ((e & 1) * 16));
    }
  }
}

hipError_t launch_kv_write(const aflex_kv_write_args& a, hipStream_t stream) {
  if (a.T == 0 || a.max_seqlen == 0) return hipSuccess;
  const int slots = (a.max_seqlen + 15) / 16 + 1;
  ProfScope ps("kv_write", stream);
  kv_write_kernel<<<dim3(slots, a.B), a.Hkv * (a.D / 8), 0, stream>>>(a);
  return hipGetLastError();
}

hipError_t launch_kv_append(const aflex_kv_append_args& a, hipStream_t stream) {
  const long long n = (long long)a.B * a.Hkv * (a.D / 8);
  if (n == 0) return hipSuccess;
  ProfScope ps("kv_append", stream);
  kv_append_kernel<<<(unsigned)((n + 255) / 256), 256, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace aflex
