// One wavefront's share of paged decode attention on gfx950: single-query
// attention of the G query heads of one KV head over a run of 16-token
// blocks of one sequence (the rollout decode step the paper runs through
// vLLM's PagedAttention: Section 3.2; Appendix C, rollout generation).  Both
// schedules (pda_partition.hip, pda_stream.hip) are built from it.
//
// Mapping onto CDNA4 (64-wide wavefronts, MFMA, LDS):
//  * Tiles.  A wavefront prefetches the next block's K and V tiles (16 x D
//    bf16 each) into registers while it computes on the current one.  Every
//    tile load is a buffer load (descriptor = the tile, so no read can leave
//    it) whose instruction reads 1 KiB of contiguous memory (whole cache
//    lines) with the non-temporal hint: the cache is streamed once, and on
//    MI355X the hint lifts a plain 4 KiB-tile gather from ~6.1 to ~6.9 TB/s.
//    All K and V loads of a lane share one 32-bit offset register.
//  * Scores.  S[G][16] = Q_g K^T is one small dense contraction per block:
//    D/32 MFMA f32_16x16x32_bf16 with the G query heads (repeated to fill 16
//    rows) as the A operand and the K tile as the B operand.  The K cache
//    stores each block as D/8 chunks of [16 slots][8 elements], so the B
//    fragment of lane l in k-step c -- 8 consecutive d of token l%16, chunk
//    4c + l/16 -- is exactly the 16 bytes at offset 1024c + 16l of the tile.
//    The A operand (q) uses the same assignment of d to (k-step, k-group,
//    element), so the contraction is unchanged.
//  * Softmax.  A lane holds the scores of 4 head rows for one token.  The
//    running maximum is moved only when some score of the block exceeds it by
//    more than 2^8 (a wavefront vote); then the block max of each row is a
//    16-lane all-reduce of four DPP moves (quad swaps, half-row and row
//    mirror) and the state is rescaled.  Otherwise probabilities are taken
//    against the stale maximum (they stay below 2^8, far inside fp32), so
//    most blocks need neither the reduction nor the O rescale; the result is
//    the same softmax.  Each lane accumulates the denominator of its own
//    token column; columns are summed once, at the end.
//  * P V runs on the VALU in fp32: lane (phase, chunk) owns 8 consecutive d
//    for all G heads and the tokens of its phase; the V tile offsets that hold
//    those elements are the same 16l + 1024i as for K.  The probabilities and
//    rescale factors of a block travel from the MFMA layout to this layout
//    through LDS (double-buffered per wavefront; a wavefront barrier only).
//  * Tokens past the context in the last block are removed by selection, not
//    by multiplying with zero, so whatever those slots hold (NaN included)
//    never reaches the result.
#pragma once

#include "pda_internal.h"

namespace pda {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

template <int CTRL>
__device__ __forceinline__ float dpp_move(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// All-reduce over each row of 16 lanes; every lane of the row gets the same bits.
__device__ __forceinline__ float row16_max(float x) {
  x = fmaxf(x, dpp_move<0xB1>(x));   // quad_perm(1,0,3,2)
  x = fmaxf(x, dpp_move<0x4E>(x));   // quad_perm(2,3,0,1)
  x = fmaxf(x, dpp_move<0x141>(x));  // row_half_mirror
  x = fmaxf(x, dpp_move<0x140>(x));  // row_mirror
  return x;
}
__device__ __forceinline__ float row16_sum(float x) {
  x += dpp_move<0xB1>(x);
  x += dpp_move<0x4E>(x);
  x += dpp_move<0x141>(x);
  x += dpp_move<0x140>(x);
  return x;
}

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float readlane_f(float x, int lane) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), lane));
}

// Raw buffer resource over `bytes` bytes at `base` (gfx9 dword-3 default:
// 32-bit raw accesses, bounds-checked against num_records).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const void* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, 0x00020000);
}

// 16-byte non-temporal load (cache policy NT) at byte `offset` of a tile.
__device__ __forceinline__ uint4 load_stream(__amdgpu_buffer_rsrc_t r, int offset) {
  const u32x4_t t = __builtin_amdgcn_raw_buffer_load_b128(r, offset, 0, 2);
  return make_uint4(t[0], t[1], t[2], t[3]);
}

// Widen 8 packed bf16 (a 16-byte load) to fp32: bf16 is the top half of fp32.
__device__ __forceinline__ void unpack8(const uint4 u, float (&f)[8]) {
  f[0] = __uint_as_float(u.x << 16);
  f[1] = __uint_as_float(u.x & 0xffff0000u);
  f[2] = __uint_as_float(u.y << 16);
  f[3] = __uint_as_float(u.y & 0xffff0000u);
  f[4] = __uint_as_float(u.z << 16);
  f[5] = __uint_as_float(u.z & 0xffff0000u);
  f[6] = __uint_as_float(u.w << 16);
  f[7] = __uint_as_float(u.w & 0xffff0000u);
}

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int G, int D>
struct WaveAttention {
  static_assert(G >= 1 && G <= kMaxGroup, "query heads per KV head");
  static_assert(D == 64 || D == 128, "head_dim");
  static constexpr int NC = D / 32;               // MFMA k-steps per block
  static constexpr int CPR = D / 8;               // 16-byte chunks per V row
  static constexpr int NPH = kWaveSize / CPR;     // token phases of the P.V layout
  static constexpr int TPL = kBlockTokens / NPH;  // tokens per lane per block in P.V
  static constexpr int GP = (G + 3) & ~3;         // head count padded to float4
  static constexpr int kTileBytes = kBlockTokens * D * 2;
  static constexpr float kNegInf = -__builtin_huge_valf();
  static constexpr float kRescaleSlack = 8.f;     // log2 of the largest unnormalised probability

  // Per-wavefront LDS for the layout change MFMA -> P.V (double-buffered).
  struct Exchange {
    float p[2][kBlockTokens][GP];
    float alpha[2][GP];
  };

  Exchange* x;
  int lane, n, kg, tp;
  float scale_log2;
  bool bad;  // a block id outside the pool was met (never dereferenced)
  bf16x8_t qa[NC];
  float o[G][8];
  float m_run[4], l_run[4];

  __device__ __forceinline__ WaveAttention(Exchange* ex, float scale_log2_)
      : x(ex), scale_log2(scale_log2_), bad(false) {
    lane = threadIdx.x & (kWaveSize - 1);
    n = lane & 15;       // MFMA row of A (head) / column of B (token)
    kg = lane >> 4;      // MFMA k-group: k-step c covers d = 8 * (4c + kg) + e
    tp = lane / CPR;     // P.V: d in [8 * (lane % CPR), +8) for tokens tp, tp + NPH, ...
  }

  // Load the G query rows starting at `q_rows` (A operand, d = 32c + 8kg + e)
  // and clear the softmax state and the bad-id flag.
  __device__ __forceinline__ void start(const uint16_t* q_rows) {
    bad = false;
    const uint16_t* qrow = q_rows + (n % G) * D + kg * 8;
#pragma unroll
    for (int c = 0; c < NC; ++c)
      qa[c] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(qrow + 32 * c));
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) o[h][e] = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      m_run[i] = kNegInf;
      l_run[i] = 0.f;
    }
  }

  // Issue the K and V tile loads of one block (or, when !needed, loads through a
  // zero-length descriptor that the hardware drops without touching memory).
  __device__ __forceinline__ void load_tiles(uint4 (&kr)[NC], uint4 (&vr)[TPL], const char* kpool,
                                             const char* vpool, size_t block_bytes, int num_blocks, int phys,
                                             bool needed) {
    if ((unsigned)phys >= (unsigned)num_blocks) {  // contract violation: never read outside the pool
      bad = true;
      phys = 0;
    }
    const size_t off = (size_t)phys * block_bytes;
    const int bytes = needed ? kTileBytes : 0;
    const __amdgpu_buffer_rsrc_t rk = tile_rsrc(kpool + off, bytes);
    const __amdgpu_buffer_rsrc_t rv = tile_rsrc(vpool + off, bytes);
    const int lane_off = lane * 16;
#pragma unroll
    for (int c = 0; c < NC; ++c) kr[c] = load_stream(rk, lane_off + c * 1024);
#pragma unroll
    for (int i = 0; i < TPL; ++i) vr[i] = load_stream(rv, lane_off + i * 1024);
  }

  // Fold one block (logical tokens tok0 .. tok0+15, context length L) into the state.
  __device__ __forceinline__ void process(const uint4 (&kr)[NC], const uint4 (&vr)[TPL], int tok0, int L, int par) {
    // ---- scores: S = Q_g K^T on MFMA; lane holds rows 4*kg+i, column n ----
    floatx4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NC; ++c)
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[c], __builtin_bit_cast(bf16x8_t, kr[c]), acc, 0, 0, 0);
    const bool tail = tok0 + kBlockTokens > L;  // wave-uniform
    float sc[4];
    bool grow = false;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sc[i] = acc[i] * scale_log2;
      if (tail && tok0 + n >= L) sc[i] = kNegInf;
      grow |= sc[i] > m_run[i] + kRescaleSlack;
    }
    // ---- move the running max only when a score outgrows it by 2^8 ----
    const bool rescale = __builtin_amdgcn_ballot_w64(grow) != 0;  // wave-uniform
    float al[4] = {1.f, 1.f, 1.f, 1.f};
    if (rescale) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float mn = fmaxf(m_run[i], row16_max(sc[i]));  // finite: the block has a valid token
        al[i] = exp2_fast(m_run[i] - mn);
        l_run[i] *= al[i];
        m_run[i] = mn;
      }
    }
    float pr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      pr[i] = exp2_fast(sc[i] - m_run[i]);
      l_run[i] += pr[i];
    }
    if (4 * kg < G) {
      *reinterpret_cast<float4*>(&x->p[par][n][4 * kg]) = make_float4(pr[0], pr[1], pr[2], pr[3]);
      if (rescale && n == 0)
        *reinterpret_cast<float4*>(&x->alpha[par][4 * kg]) = make_float4(al[0], al[1], al[2], al[3]);
    }
    wave_lds_sync();

    // ---- O = alpha * O + P V on the VALU ----
    if (rescale) {
      float alpha[GP];
#pragma unroll
      for (int h4 = 0; h4 < GP; h4 += 4) {
        const float4 t = *reinterpret_cast<const float4*>(&x->alpha[par][h4]);
        alpha[h4] = t.x; alpha[h4 + 1] = t.y; alpha[h4 + 2] = t.z; alpha[h4 + 3] = t.w;
      }
#pragma unroll
      for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) o[h][e] *= alpha[h];
    }
#pragma unroll
    for (int i = 0; i < TPL; ++i) {
      const int row = i * NPH + tp;
      float f[8];
      unpack8(vr[i], f);
      if (tail && tok0 + row >= L) {
#pragma unroll
        for (int e = 0; e < 8; ++e) f[e] = 0.f;
      }
      float ph[GP];
#pragma unroll
      for (int h4 = 0; h4 < GP; h4 += 4) {
        const float4 t = *reinterpret_cast<const float4*>(&x->p[par][row][h4]);
        ph[h4] = t.x; ph[h4 + 1] = t.y; ph[h4 + 2] = t.z; ph[h4 + 3] = t.w;
      }
#pragma unroll
      for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) o[h][e] = fmaf(ph[h], f[e], o[h][e]);
    }
  }

  // Stream blocks [j0, j1) of one sequence: block ids in `table_row`, tiles of
  // this KV head at kpool/vpool + id * block_bytes, context length L.
  //
  // Two register buffers: the tiles of block i+1 are in flight while block i
  // is computed.  Every load is unconditional, so the compiler counts
  // outstanding loads exactly and waits only for the tiles it is about to
  // use; the scheduling barriers keep each prefetch ahead of the first use of
  // the current tiles.  Past the end of the run the prefetch gets a
  // zero-length descriptor.  Block ids come 64 at a time, one per lane, and
  // are read with readlane, so no tile load waits on a scalar load.
  __device__ __forceinline__ void run(const int32_t* table_row, int j0, int j1, int L, const char* kpool,
                                      const char* vpool, size_t block_bytes, int num_blocks) {
    const int cnt = j1 - j0;
    uint4 k0[NC], v0[TPL], k1[NC], v1[TPL];
    for (int c0 = 0; c0 < cnt; c0 += kWaveSize) {
      const int cn = min(kWaveSize, cnt - c0);
      const int jc = j0 + c0;
      const int ids = lane < cn ? table_row[jc + lane] : 0;
      auto id = [&](int i) { return __builtin_amdgcn_readlane(ids, i); };
      load_tiles(k0, v0, kpool, vpool, block_bytes, num_blocks, id(0), true);
      for (int i = 0; i < cn; i += 2) {
        load_tiles(k1, v1, kpool, vpool, block_bytes, num_blocks, id(min(i + 1, cn - 1)), i + 1 < cn);
        __builtin_amdgcn_sched_barrier(0);
        process(k0, v0, (jc + i) * kBlockTokens, L, 0);
        if (i + 1 >= cn) break;
        load_tiles(k0, v0, kpool, vpool, block_bytes, num_blocks, id(min(i + 2, cn - 1)), i + 2 < cn);
        __builtin_amdgcn_sched_barrier(0);
        process(k1, v1, (jc + i + 1) * kBlockTokens, L, 1);
      }
    }
  }

  // Reduce the per-lane state: denominators over the 16 token columns of each
  // row, O over the token phases.  Afterwards lanes < CPR hold O[h][8*lane + e]
  // for every head h < G, and every lane holds each head's max mh[h] and
  // denominator lh[h] (head h sits in MFMA row h: k-group h/4, register h%4).
  float mh[G], lh[G];
  __device__ __forceinline__ void finish() {
#pragma unroll
    for (int i = 0; i < 4; ++i) l_run[i] = row16_sum(l_run[i]);
#pragma unroll
    for (int h = 0; h < G; ++h) {
      mh[h] = readlane_f(m_run[h & 3], 16 * (h >> 2));
      lh[h] = readlane_f(l_run[h & 3], 16 * (h >> 2));
    }
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e)
#pragma unroll
        for (int s = CPR; s < kWaveSize; s <<= 1) o[h][e] += __shfl_xor(o[h][e], s);
  }
};

}  // namespace pda
