// Batched GQA decode attention over a paged bf16 KV cache, gfx950.
//
// Operation: for every sequence b and query head h, softmax-weighted sum of
// the cached values of kv head g = h / G over the ctx_b cached tokens, the
// decode-step attention the paper treats as the memory-bound operator
// (section 1; section 3.2).
//
// Design (HBM-bound: every cached K/V byte is read exactly once, in one
// launch):
//  * Work partition. The (sequence, kv head) units are laid end to end in
//    (b, kv head) order, each as its ceil(ctx_b / 16) blocks plus a fixed
//    charge for the piece it adds; the work-groups take consecutive ranges of
//    that flattened range in work-group order: equal ones (or a fixed size
//    the caller asks for), except that in the grid of three work-groups per
//    CU of a call that has the GPU to itself the three dispatch rounds take
//    ranges weighted 5:3:1, since the first work-group dispatched to a CU
//    progresses fastest. Every work-group
//    computes the partition itself from the context lengths (no host
//    synchronisation, no extra launch); a work-group's range is one or more
//    pieces, each the part of one unit that falls into it. The grid is the
//    resident work-groups: three 4-wave ones per CU, or one 12-wave one per
//    CU for calls beside other GPU work. Short contexts take one work-group
//    per unit instead.
//  * Piece kernel body: the waves take pairs of 16-token blocks round-robin.
//    Per pair a wave issues 16 (D=128) 16-byte loads per lane straight into
//    MFMA operand registers -- no LDS staging is needed because both
//    contractions see their operand with the contraction index contiguous:
//      S^T[tok][g] = K[tok][:] . q[g][:]       (v_mfma_f32_16x16x32_bf16,
//                                               K rows = 16 tokens, 16 cols = G
//                                               query heads padded to 16)
//      O^T[d][g]  += V^T[d][tok] . P^T[tok][g]  (V pool is [.., D, 16] so 8
//                                               consecutive tokens of one d are
//                                               one 16-byte load)
//    The token order inside the QK tile is chosen so that the S^T output
//    registers of a lane are exactly the P^T operand registers it needs for
//    the PV product, and all softmax state of head g lives in the four lanes
//    with lane % 16 == g: the online softmax needs two cross-lane max steps per
//    block pair and no LDS round trip. At a piece's end each wave deposits
//    its partial in an LDS slot (a ring of two for G <= 8) and goes on to the
//    next piece; the wave that deposits last merges the piece's partials in
//    wave order, so no wave waits at a barrier for the one with an extra pair
//    and the result does not depend on which wave merges.
//  * Merge. A unit held by one piece writes its bf16 output directly. A unit
//    cut into several pieces (consecutive work-groups; only the first and the
//    last piece of a work-group's range can be such a piece) has each piece
//    write an fp32 partial (O, m, l) to slot unit + work-group, unique over
//    all pieces; a second, small launch merges the partials of those units in
//    work-group order. Exchanging partials inside the first launch (flags or
//    tickets between work-groups, each a round trip through the loaded
//    memory system) stalled the work-groups that hold split units by several
//    microseconds per exchange, more than the second launch costs.
#include <math.h>

#include <atomic>

#include "common.h"
#include "kernels.h"
#include "profile.h"

namespace aflex {

struct AttnParams {
  const uint16_t* q;
  const uint16_t* kc;
  const uint16_t* vc;
  const int32_t* bt;
  const int32_t* cl;
  uint16_t* out;
  float* part_o;                 // [U + P][G][D]
  float* part_ml;                // [U + P][G][2]  (running max in log2 units, sum)
  int2* span;                    // [U]  first and last work-group of each unit's pieces
  int B, Hq, Hkv, G;
  int max_blocks, num_blocks, max_ctx;
  int chunk_blocks;              // > 0: fixed blocks per work-group; 0: even split over the grid
  int unit_cost;                 // extra cost of a unit in block positions (0 with fixed pieces)
  int rounds;                    // 3: range sizes weighted by dispatch round (see split_of); else 1
  float scale_log2;              // softmax scale * log2(e)
};

constexpr int kWaves = 4;
constexpr int kMinChunkBlocks = 8;  // one pair per wave at least
// Charge per (sequence, kv head) unit, in 16-token blocks, when the grid
// splits the units evenly: a piece costs its work-group about one loaded round
// trip to memory besides its blocks (the waves drain at its end, the merge
// through LDS runs, the next piece's first loads start cold), so work-groups
// covering many short units get fewer blocks.
constexpr int kUnitCost = 8;

__device__ __forceinline__ int clamp_ctx(const AttnParams& p, int b) {
  int c = p.cl[b];
  return c < 0 ? 0 : (c > p.max_ctx ? p.max_ctx : c);
}

__device__ __forceinline__ int nblk_of(int ctx) { return (ctx + 15) >> 4; }

// K/V tile loads; NT marks them non-temporal (each cached byte is read once).
template <bool NT>
__device__ __forceinline__ bf16x8 ld_kv(const uint16_t* ptr) {
  if constexpr (NT) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    return __builtin_bit_cast(bf16x8, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(ptr)));
  } else {
    return ld_bf16x8(ptr);
  }
}

__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ int wave_incl_scan(int v, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(v, o);
    if (lane >= o) v += t;
  }
  return v;
}

// Block id of local block jb of sequence b's table, or -1 when jb is past the
// piece's end or the table entry is out of range (its tokens are masked).
__device__ __forceinline__ int load_block_id(const AttnParams& p, int b, int jb, int j_end) {
  int id = -1;
  if (jb < j_end) {
    id = p.bt[(size_t)b * p.max_blocks + jb];
    if (id < 0 || id >= p.num_blocks) id = -1;
  }
  return id;
}

// Positions a (sequence, kv head) unit of sequence b takes in the flattened
// range: its blocks plus a fixed charge for the piece it adds (zero for a
// sequence with no cached token, which has no unit).
__device__ __forceinline__ int unit_len(const AttnParams& p, int b) {
  const int n = nblk_of(clamp_ctx(p, b));
  return n > 0 ? n + p.unit_cost : 0;
}

// Partition of the flattened range, as the decode kernel computes it: the
// total over all units (W) and the positions per work-group.
__device__ __forceinline__ int chunk_of(const AttnParams& p, int P, int lane, int* W_out) {
  int total = 0;
  for (int c = 0; c < p.B; c += 64) {
    const int b = c + lane;
    total += wave_sum_i(b < p.B ? unit_len(p, b) : 0);
  }
  const int W = __builtin_amdgcn_readfirstlane(total) * p.Hkv;
  *W_out = W;
  return p.chunk_blocks ? p.chunk_blocks : max((W + P - 1) / P, kMinChunkBlocks);
}

// Relative range sizes of the three work-groups that share a CU in the
// resident grid, by dispatch round (work-groups [0, P/3) are dispatched
// first, one per CU, then the next P/3). With equal ranges the first
// work-group on a CU ends first and the third last (Qwen3-32B B = 64: 35.7,
// 44.2 and 52.0 us on average, the same placement and order in every run):
// the older waves win the CU's arbitration. Weighting the ranges by round
// shortens the launch (Qwen3-32B B = 64, uniform / 6:5:4 / 4:3:2 / 5:3:1 /
// 6:3:1 / 3:2:0: 63.3 / 63.1 / 62.4 / 61.8 / 61.8 / 63.1 us; long-context
// B = 256: 871 -> 868 us with 5:3:1).
constexpr int kRoundWeight[3] = {5, 3, 1};

// Ranges of the work-groups: wg = k R + i (round k < rounds, 0 <= i < R) takes
// c_k positions, the ranges laid end to end in work-group order. (Plain
// scalars, not a struct: a struct here was kept in per-thread LDS copies.)
__device__ __forceinline__ void split_of(const AttnParams& p, int P, int W, int C, int& R, int& c0, int& c1,
                                         int& c2) {
  if (p.rounds == 3 && p.chunk_blocks == 0) {
    // rounds 0 and 1 from the weights, round 2 the rest (so the ranges cover W)
    R = P / 3;
    const float per = (float)W / (float)(R * (kRoundWeight[0] + kRoundWeight[1] + kRoundWeight[2]));
    c0 = max((int)(per * kRoundWeight[0]), kMinChunkBlocks);
    c1 = max((int)(per * kRoundWeight[1]), kMinChunkBlocks);
    const int rest = W - R * (c0 + c1);
    c2 = max((rest + R - 1) / R, kMinChunkBlocks);
  } else {
    R = P;
    c0 = c1 = c2 = C;
  }
  R = __builtin_amdgcn_readfirstlane(R);
  c0 = __builtin_amdgcn_readfirstlane(c0);
  c1 = __builtin_amdgcn_readfirstlane(c1);
  c2 = __builtin_amdgcn_readfirstlane(c2);
}

__device__ __forceinline__ int split_start(int R, int c0, int c1, int c2, int wg) {
  const int k = wg / R;
  const int i = wg - k * R;
  return (k > 0 ? R * c0 : 0) + (k > 1 ? R * c1 : 0) + i * (k == 0 ? c0 : k == 1 ? c1 : c2);
}

__device__ __forceinline__ int split_size(int R, int c0, int c1, int c2, int wg) {
  const int k = wg / R;
  return k == 0 ? c0 : k == 1 ? c1 : c2;
}

// Work-group whose range holds position x (x below the total).
__device__ __forceinline__ int split_owner(int R, int c0, int c1, int c2, int x) {
  const int e0 = R * c0;
  if (x < e0) return x / c0;
  const int e1 = e0 + R * c1;
  if (x < e1) return R + (x - e0) / c1;
  return 2 * R + (x - e1) / c2;
}

// UNIT: one work-group per (sequence, kv head) unit, written whole (no
// partials); otherwise the even split of the flattened range.
template <int D, bool NT, bool UNIT, int NW = kWaves>
__global__ __launch_bounds__(64 * NW, 12 / NW) void attn_decode_kernel(AttnParams p) {
  constexpr int NC = D / 32;   // k-chunks of the QK product
  constexpr int NMT = D / 16;  // d-tiles of the PV product
  constexpr int LDO = D + 4;   // padded row of the LDS merge buffer

  constexpr int NT_ = 64 * NW;  // threads
  // Piece partials of the waves, in a ring of LDS slots: two slots of 8 head
  // rows per wave when G <= 8, else one slot of 16 rows (the same bytes).
  // Per slot, arrive counts the waves that deposited the current piece and
  // gen counts the pieces merged out of it.
  __shared__ float sm_ml[NW * 16 * 2];
  __shared__ __attribute__((aligned(16))) float sm_o[NW * 16 * LDO];
  __shared__ int sm_arrive[2];
  __shared__ int sm_gen[2];

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int r = lane & 15;   // MFMA row/col within the 16-wide tile
  const int qg = lane >> 4;  // lane group: which 8-wide k slice the lane feeds
  const int G = p.G;
  const int Hkv = p.Hkv;
  const int wg = blockIdx.x;
  const int P = gridDim.x;
  const int GR = G <= 8 ? 8 : 16;     // head rows of a slot
  const int nslot = G <= 8 ? 2 : 1;

  if (tid < 2) {
    sm_arrive[tid] = 0;
    sm_gen[tid] = 0;
  }
  __syncthreads();

  // Sequences with no cached token produce zeros; work-group wg clears those
  // with b = wg (mod P).
  for (int b = wg; b < p.B; b += P) {
    if (clamp_ctx(p, b) == 0) {
      uint4* o = reinterpret_cast<uint4*>(p.out + (size_t)b * p.Hq * D);
      for (int i = tid; i < p.Hq * D / 8; i += NT_) o[i] = make_uint4(0, 0, 0, 0);
    }
  }

  // ---- partition: this work-group's range of the flattened blocks ----
  // (UNIT: work-group wg takes unit wg = (sequence ub, kv head wg % Hkv), all
  // of its blocks as one piece, with a chunk no range can span twice.)
  int W = 0;
  int sR = P, sc0 = 1 << 30, sc1 = 1 << 30, sc2 = 1 << 30;
  if constexpr (!UNIT) {
    const int C = chunk_of(p, P, lane, &W);
    if constexpr (NW == kWaves) {  // the grid of three work-groups per CU
      split_of(p, P, W, C, sR, sc0, sc1, sc2);
    } else {
      sc0 = sc1 = sc2 = C;
    }
  }
  const int ub = UNIT ? wg / Hkv : 0;
  const int unb = UNIT ? (ub < p.B ? nblk_of(clamp_ctx(p, ub)) : 0) : 0;
  const int x0 = __builtin_amdgcn_readfirstlane(UNIT ? (wg - ub * Hkv) * unb : split_start(sR, sc0, sc1, sc2, wg));
  if (UNIT ? unb == 0 : x0 >= W) return;
  const int x1 = __builtin_amdgcn_readfirstlane(UNIT ? x0 + unb : min(x0 + split_size(sR, sc0, sc1, sc2, wg), W));

  // First sequence whose units reach past x0: base = its first position per
  // kv head. Unit (b, kvh) spans positions [S, S + len) with
  // S = base * Hkv + kvh * len and len = nblk + unit_cost; its block j sits at
  // S + unit_cost + j, so a work-group whose range lies in a unit's leading
  // charge holds no piece of it.
  int b = ub, base = 0;
  if constexpr (!UNIT) {
    for (int c = 0; c < p.B; c += 64) {
      const int bb = c + lane;
      const int n = bb < p.B ? unit_len(p, bb) : 0;
      const int incl = wave_incl_scan(n, lane);
      const unsigned long long past = __ballot((base + incl) * Hkv > x0);
      if (past) {
        const int l = __builtin_ctzll(past);
        b = c + l;
        base += __builtin_amdgcn_readlane(incl - n, l);
        break;
      }
      base += __builtin_amdgcn_readlane(incl, 63);
    }
  }
  // (every value that steers the piece loop is wave-uniform: scalar registers)
  b = __builtin_amdgcn_readfirstlane(b);
  base = __builtin_amdgcn_readfirstlane(base);
  const int uc = UNIT ? 0 : p.unit_cost;
  int nb = nblk_of(clamp_ctx(p, b));
  int kvh = (x0 - base * Hkv) / (nb + uc);

  // Token slots. QK tile row rr (lane rr loads it) holds token
  //   block (rr >> 3), offset ((rr >> 2) & 1) * 8 + (rr & 3)    [first product]
  //   ... + 4                                                  [second product]
  // so output rows 4*qg + i of the two products are tokens (qg&1)*8 + i and
  // (qg&1)*8 + 4 + i of block (qg >> 1): the 8 consecutive tokens whose V^T
  // slice this lane loads for the PV product.
  const int ksel = r >> 3;
  const int ktok = ((r >> 2) & 1) * 8 + (r & 3);
  const int vsel = qg >> 1;
  const int vtok = (qg & 1) * 8;

  int rot = 0;  // wave that takes the piece's first pair: spreads the odd pairs over the waves

  int x = x0;
  int piece = 0;  // pieces this work-group has finished
  // First block-id chunk of the current piece; each piece loads the next
  // piece's first chunk while it streams, so a new piece starts with its K/V
  // loads instead of a round trip for its block ids.
  int piece_ids;
  {
    const int us = base * Hkv + kvh * (nb + uc) + uc;
    piece_ids = load_block_id(p, b, max(x0 - us, 0) + lane, min(nb, x1 - us));
  }
  while (x < x1) {
    const int ctx = clamp_ctx(p, b);
    const int ustart = base * Hkv + kvh * (nb + uc) + uc;  // position of the unit's first block
    const int j0 = max(x - ustart, 0);
    const int j1 = min(nb, x1 - ustart);
    const int h0 = kvh * G;
    const int npairs = (j1 - j0 + 1) / 2;

    // The next unit (its range starts where this piece ends when the piece
    // reaches the unit's last block): the next kv head of b, else the next
    // sequence with blocks. A range that ends inside this unit, or inside its
    // leading charge (j1 <= 0), ends the loop.
    const int xn = ustart + max(j1, 0);
    int bn = b, kvhn = kvh + 1, basen = base, nbn = nb;
    if (kvhn == Hkv) {
      kvhn = 0;
      basen = base + nb + uc;
      do {
        ++bn;
      } while (xn < x1 && bn < p.B && nblk_of(clamp_ctx(p, bn)) == 0);
      nbn = (xn < x1) ? nblk_of(clamp_ctx(p, bn)) : 0;
    }
    const int next_piece_ids = (xn < x1) ? load_block_id(p, bn, lane, min(nbn, x1 - xn - uc)) : -1;
    if (j1 <= j0) break;  // the range ends inside the unit's leading charge

    // q as the B operand of the QK product: column g = r, k = d in [c*32 + qg*8, +8).
    bf16x8 qf[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      qf[c] = (r < G) ? ld_bf16x8(p.q + ((size_t)b * p.Hq + h0 + r) * D + c * 32 + qg * 8)
                      : zero_bf16x8();
    }

    // Block ids of the piece, 64 per wave register (lane l: local block
    // j0 + 64 c + l of chunk c); the next chunk is loaded one chunk ahead.
    int my_id = piece_ids;
    int next_id = (npairs > 32) ? load_block_id(p, b, j0 + 64 + lane, j1) : -1;
    int cur_chunk = 0;

    float m_run = kNegInf;
    float l_run = 0.f;
    f32x4 acc[NMT];
#pragma unroll
    for (int mt = 0; mt < NMT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int pr = (int)((unsigned)(wave - rot + NW) % NW); pr < npairs; pr += NW) {
      if ((pr >> 5) != cur_chunk) {  // advances by at most one chunk per step
        cur_chunk = pr >> 5;
        my_id = next_id;
        next_id = ((cur_chunk + 1) * 32 < npairs) ? load_block_id(p, b, j0 + (cur_chunk + 1) * 64 + lane, j1) : -1;
      }
      const int idA = __builtin_amdgcn_readlane(my_id, (2 * pr) & 63);
      const int idB = __builtin_amdgcn_readlane(my_id, (2 * pr + 1) & 63);
      const int tA = (j0 + 2 * pr) * 16;

      bf16x8 k1[NC], k2[NC], vf[NMT];
      const int pk = ksel ? idB : idA;
      if (pk >= 0) {
        const uint16_t* kb = p.kc + ((size_t)pk * Hkv + kvh) * 16 * D + qg * 8;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          k1[c] = ld_kv<NT>(kb + ktok * D + c * 32);
          k2[c] = ld_kv<NT>(kb + (ktok + 4) * D + c * 32);
        }
      } else {
#pragma unroll
        for (int c = 0; c < NC; ++c) k1[c] = k2[c] = zero_bf16x8();
      }
      const int pv = vsel ? idB : idA;
      const int tb = tA + vsel * 16 + vtok;  // first token of this lane's 8-token slice
      const int nv = (pv >= 0) ? ctx - tb : 0;
      if (pv >= 0) {
        const uint16_t* vb = p.vc + ((size_t)pv * Hkv + kvh) * D * 16 + vtok;
#pragma unroll
        for (int mt = 0; mt < NMT; ++mt) vf[mt] = ld_kv<NT>(vb + (mt * 16 + r) * 16);
      } else {
#pragma unroll
        for (int mt = 0; mt < NMT; ++mt) vf[mt] = zero_bf16x8();
      }
      if (nv < 8) {  // tail of the last block (or a skipped block): zero V so 0 * NaN cannot leak
#pragma unroll
        for (int mt = 0; mt < NMT; ++mt) vf[mt] = keep_first(vf[mt], nv);
      }

      f32x4 s1 = {0.f, 0.f, 0.f, 0.f}, s2 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1[c], qf[c], s1, 0, 0, 0);
        s2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k2[c], qf[c], s2, 0, 0, 0);
      }

      float sv[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        sv[i] = (i < nv) ? s1[i] * p.scale_log2 : kNegInf;
        sv[4 + i] = (4 + i < nv) ? s2[i] * p.scale_log2 : kNegInf;
      }
      float mx = sv[0];
#pragma unroll
      for (int i = 1; i < 8; ++i) mx = fmaxf(mx, sv[i]);
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx);
      const float m_use = (m_new == kNegInf) ? 0.f : m_new;
      const float alpha = fast_exp2(m_run - m_use);
      bf16x8 pb;
      float ps = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const __bf16 e = static_cast<__bf16>(fast_exp2(sv[i] - m_use));
        pb[i] = e;
        ps += static_cast<float>(e);
      }
      l_run = l_run * alpha + ps;
      m_run = m_new;
#pragma unroll
      for (int mt = 0; mt < NMT; ++mt) {
        acc[mt] *= alpha;
        acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[mt], pb, acc[mt], 0, 0, 0);
      }
    }

    // Sum of the softmax denominators over the 4 lanes that share head g.
    l_run += __shfl_xor(l_run, 16);
    l_run += __shfl_xor(l_run, 32);

    // Deposit this wave's partial in the piece's slot once the slot's previous
    // piece has been merged out of it; the wave that deposits last merges the
    // piece. No wave waits for the others at a piece boundary: the ones done
    // with their pairs go on to the next piece's loads.
    const int slot = piece & (nslot - 1);
    const int use = piece / nslot;
    while (__hip_atomic_load(&sm_gen[slot], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) != use)
      __builtin_amdgcn_s_sleep(1);
    float* so = sm_o + (slot * NW * GR) * LDO;
    float* sml = sm_ml + slot * NW * GR * 2;
    if (r < G) {
      if (qg == 0) {
        sml[(wave * GR + r) * 2 + 0] = m_run;
        sml[(wave * GR + r) * 2 + 1] = l_run;
      }
#pragma unroll
      for (int mt = 0; mt < NMT; ++mt)
        *reinterpret_cast<f32x4*>(&so[(wave * GR + r) * LDO + mt * 16 + 4 * qg]) = acc[mt];
    }
    int arrived = 0;
    if (lane == 0)
      arrived = __hip_atomic_fetch_add(&sm_arrive[slot], 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_WORKGROUP);
    arrived = __builtin_amdgcn_readfirstlane(arrived);

    if (arrived == NW - 1) {
      // Work-groups holding pieces of this unit; the one with its first piece
      // records the span for the merge launch.
      const int wg_first = UNIT ? 0 : split_owner(sR, sc0, sc1, sc2, ustart);
      const int wg_last = UNIT ? 0 : split_owner(sR, sc0, sc1, sc2, ustart + nb - 1);
      const int unit = b * Hkv + kvh;
      const size_t seg = (size_t)unit + wg;
      if (lane == 0 && wg == wg_first) p.span[unit] = make_int2(wg_first, wg_last);

      constexpr int D4 = D / 4;
      for (int it = lane; it < G * D4; it += 64) {
        const int g = it / D4;
        const int d4 = it - g * D4;
        float M = sml[g * 2];
#pragma unroll
        for (int w = 1; w < NW; ++w) M = fmaxf(M, sml[(w * GR + g) * 2]);
        const float Mu = (M == kNegInf) ? 0.f : M;
        float L = 0.f;
        f32x4 O = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 2
        for (int w = 0; w < NW; ++w) {
          const float wt = fast_exp2(sml[(w * GR + g) * 2] - Mu);
          L += wt * sml[(w * GR + g) * 2 + 1];
          O += wt * *reinterpret_cast<const f32x4*>(&so[(w * GR + g) * LDO + d4 * 4]);
        }
        if (wg_first == wg_last) {
          ushort4 v;
          v.x = f2bf(L > 0.f ? O[0] / L : 0.f);
          v.y = f2bf(L > 0.f ? O[1] / L : 0.f);
          v.z = f2bf(L > 0.f ? O[2] / L : 0.f);
          v.w = f2bf(L > 0.f ? O[3] / L : 0.f);
          *reinterpret_cast<ushort4*>(p.out + ((size_t)b * p.Hq + h0 + g) * D + d4 * 4) = v;
        } else {
          *reinterpret_cast<f32x4*>(&p.part_o[(seg * G + g) * D + d4 * 4]) = O;
          if (d4 == 0) {
            p.part_ml[(seg * G + g) * 2 + 0] = M;
            p.part_ml[(seg * G + g) * 2 + 1] = L;
          }
        }
      }
      // The slot is free again once every read of it above is done.
      if (lane == 0) {
        sm_arrive[slot] = 0;
        __hip_atomic_store(&sm_gen[slot], use + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
    }
    ++piece;

    rot = (int)((unsigned)(rot + npairs) % NW);

    x = xn;
    b = bn;
    kvh = kvhn;
    base = basen;
    nb = nbn;
    piece_ids = next_piece_ids;
  }
}

// Merge launch: work-group u merges unit u (sequence b = u / Hkv, kv head
// u % Hkv) if the decode launch split it between work-groups (the span its
// first piece recorded); each thread combines 4 consecutive d of one head
// over the pieces in work-group order.
template <int D>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnParams p) {
  constexpr int D4 = D / 4;
  const int unit = blockIdx.x;
  const int b = unit / p.Hkv, kvh = unit - b * p.Hkv;
  if (clamp_ctx(p, b) == 0) return;  // no piece, no recorded span
  const int2 sp = p.span[unit];
  const int wf = sp.x, wl = sp.y;
  if (wf == wl) return;  // written by the decode launch
  const int G = p.G;
  for (int it = threadIdx.x; it < G * D4; it += 256) {
    const int g = it / D4;
    const int d4 = it - g * D4;
    // One pass over the pieces with a running maximum: every piece's loads are
    // independent of the running state, so they go out together.
    float M = kNegInf, L = 0.f;
    f32x4 O = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (int w = wf; w <= wl; ++w) {
      const size_t s = (size_t)unit + w;
      const float m = p.part_ml[(s * G + g) * 2];
      const float l = p.part_ml[(s * G + g) * 2 + 1];
      const f32x4 o = *reinterpret_cast<const f32x4*>(&p.part_o[(s * G + g) * D + d4 * 4]);
      const float Mn = fmaxf(M, m);
      const float Mu = (Mn == kNegInf) ? 0.f : Mn;
      const float wa = fast_exp2(M - Mu);  // weight of the pieces so far
      const float wb = fast_exp2(m - Mu);  // weight of piece w
      L = L * wa + l * wb;
      O = O * wa + o * wb;
      M = Mn;
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    ushort4 v;
    v.x = f2bf(O[0] * inv);
    v.y = f2bf(O[1] * inv);
    v.z = f2bf(O[2] * inv);
    v.w = f2bf(O[3] * inv);
    *reinterpret_cast<ushort4*>(p.out + ((size_t)b * p.Hq + kvh * G + g) * D + d4 * 4) = v;
  }
}

// ---------------------------------------------------------------------------
// Host side.

// Work-groups resident at once: three 4-wave work-groups per CU (the kernel's
// register budget allows three waves per SIMD; two or four per CU measured
// slower on the Qwen3-32B B = 64 workload: 69.9 and 75.4 against 65.5 us).
static int resident_wgs() {
  static std::atomic<int> cached{0};
  int v = cached.load(std::memory_order_relaxed);
  if (v > 0) return v;
  int dev = 0, ncu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || ncu <= 0)
    ncu = 256;
  v = 3 * ncu;
  cached.store(v, std::memory_order_relaxed);
  return v;
}

// Waves of the work-groups of the even split when it runs beside other work
// on the GPU (the pipeline step): one 12-wave work-group per CU, its LDS
// merge buffers (103 KiB) leaving a CU to either attention or FFN work. Alone,
// three 4-wave work-groups per CU are faster (Qwen3-32B B = 64: 63.2 against
// 63.9 us); beside the FFN stream the wide form took the pipeline step from
// 2.71 to 2.67 ms. The layer step, whose attention stream also runs o_proj,
// is faster with the 4-wave form (2.742 against 2.768 ms).
constexpr int kWideWaves = 12;

static int unit_cost(const aflex_attn_args& a) { return a.split_tokens > 0 ? 0 : kUnitCost; }

static long long work_bound(const aflex_attn_args& a) {
  return (long long)a.B * a.Hkv * ((a.max_context_len + 15) / 16 + unit_cost(a));
}

// Contexts of at most this many tokens take one work-group per (sequence, kv
// head) unit when the units fit in one round of resident work-groups: each
// unit is written directly (no partials) and the merge launch, which at these
// sizes costs more than the imbalance between units, is skipped.
constexpr int kUnitPerWgMaxCtx = 512;

static bool unit_per_wg(const aflex_attn_args& a) {
  return a.split_tokens == 0 && a.max_context_len <= kUnitPerWgMaxCtx && (long long)a.B * a.Hkv <= resident_wgs();
}

// Grid size: one work-group per unit for short contexts (above); with a fixed
// piece size, enough work-groups for the bound on the blocks; otherwise the
// resident work-groups, fewer when the bound cannot give each of them a pair
// per wave.
static int attn_grid(const aflex_attn_args& a, bool wide = false) {
  if (unit_per_wg(a)) return a.B * a.Hkv > 0 ? a.B * a.Hkv : 1;
  const long long wb = work_bound(a);
  long long P;
  if (a.split_tokens > 0) {
    P = (wb + a.split_tokens / 16 - 1) / (a.split_tokens / 16);
  } else if (wide) {  // one wide work-group per CU, a pair per wave at least
    const int ncu = resident_wgs() / 3;
    P = (wb + kMinChunkBlocks * 3 - 1) / (kMinChunkBlocks * 3);
    P = P < ncu ? P : ncu;
  } else {
    P = (wb + kMinChunkBlocks - 1) / kMinChunkBlocks;
    P = P < resident_wgs() ? P : resident_wgs();
  }
  return (int)(P < 1 ? 1 : P);
}

bool attn_shape_fits(const aflex_attn_args& a) { return work_bound(a) < (1ll << 30); }

// (sized for the narrow grid, which is never smaller than the wide one)
size_t attn_workspace_bytes(const aflex_attn_args& a) {
  const size_t U = (size_t)a.B * a.Hkv;
  const size_t segs = U + (size_t)attn_grid(a);
  const size_t G = (size_t)(a.Hq / a.Hkv);
  return align_up(segs * G * a.D * sizeof(float), 256) + align_up(segs * G * 2 * sizeof(float), 256) +
         align_up(U * sizeof(int2), 256);
}

hipError_t launch_attn_decode(const aflex_attn_args& a, void* ws, hipStream_t stream, AttnForm form) {
  AttnParams p;
  p.q = a.q;
  p.kc = a.k_cache;
  p.vc = a.v_cache;
  p.bt = a.block_table;
  p.cl = a.context_lens;
  p.out = a.out;
  p.B = a.B;
  p.Hq = a.Hq;
  p.Hkv = a.Hkv;
  p.G = a.Hq / a.Hkv;
  p.max_blocks = a.max_blocks_per_seq;
  p.num_blocks = a.num_blocks;
  p.max_ctx = a.max_context_len;
  p.chunk_blocks = a.split_tokens > 0 ? a.split_tokens / 16 : 0;
  p.unit_cost = unit_cost(a);
  const bool unit = unit_per_wg(a);
  const bool wide = form == AttnForm::kWide && !unit && a.split_tokens == 0;
  const float scale = a.scale != 0.f ? a.scale : 1.0f / sqrtf((float)a.D);
  p.scale_log2 = scale * kLog2e;
  const int P = attn_grid(a, wide);
  // weighted rounds for the full grid of three 4-wave work-groups per CU
  // (beside other work the dispatch order no longer places the rounds: the
  // layer step, whose attention runs beside the MoE stream, took 2.78 ms with
  // the weighting and 2.75 ms without)
  p.rounds = (form == AttnForm::kAlone && !unit && a.split_tokens == 0 && P == resident_wgs() && P % 3 == 0) ? 3 : 1;
  const size_t U = (size_t)a.B * a.Hkv;
  const size_t segs = U + (size_t)P;
  const size_t G = (size_t)p.G;
  char* w = static_cast<char*>(ws);
  p.part_o = reinterpret_cast<float*>(w);
  w += align_up(segs * G * a.D * sizeof(float), 256);
  p.part_ml = reinterpret_cast<float*>(w);
  w += align_up(segs * G * 2 * sizeof(float), 256);
  p.span = reinterpret_cast<int2*>(w);
  {
    ProfScope ps("attn_decode", stream);
    if (a.D == 128) {
      if (unit)
        attn_decode_kernel<128, true, true><<<P, 256, 0, stream>>>(p);
      else if (wide)
        attn_decode_kernel<128, true, false, kWideWaves><<<P, 64 * kWideWaves, 0, stream>>>(p);
      else
        attn_decode_kernel<128, true, false><<<P, 256, 0, stream>>>(p);
    } else {
      if (unit)
        attn_decode_kernel<64, true, true><<<P, 256, 0, stream>>>(p);
      else if (wide)
        attn_decode_kernel<64, true, false, kWideWaves><<<P, 64 * kWideWaves, 0, stream>>>(p);
      else
        attn_decode_kernel<64, true, false><<<P, 256, 0, stream>>>(p);
    }
  }
  if (P > 1 && !unit) {  // with one work-group, or one per unit, no unit is split
    ProfScope ps("attn_merge", stream);
    if (a.D == 128)
      attn_merge_kernel<128><<<a.B * a.Hkv, 256, 0, stream>>>(p);
    else
      attn_merge_kernel<64><<<a.B * a.Hkv, 256, 0, stream>>>(p);
  }
  return hipGetLastError();
}

}  // namespace aflex
