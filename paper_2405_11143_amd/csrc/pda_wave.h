// One wavefront's share of paged attention on gfx950: up to 16 query rows --
// the G query heads of one KV head, for one or several new tokens of one
// sequence -- over a run of 16-token blocks of that sequence's context (the
// rollout decode step the paper runs through vLLM's PagedAttention, and its
// multi-token form for speculative decoding and chunked prefill: Section
// 3.2; Appendix C, rollout generation).  The partition kernel
// (pda_partition.hip) is built from it.
//
// Mapping onto CDNA4 (64-wide wavefronts, MFMA):
//  * Lanes.  Lane l = 16 kg + n works for query row n (rows past the last
//    real one repeat real rows) and, in each block, for tokens 4kg .. 4kg+3.
//    Everything a query row needs -- its running max, its denominator, its
//    rescale factor and its output -- lives in the four lanes n, n+16, n+32,
//    n+48, so the softmax needs no exchange through LDS.
//  * Tiles.  A wavefront prefetches the next block's K and V tiles (16 x D
//    bf16 each) into registers while it computes on the current one.  Every
//    tile load is a buffer load (descriptor = the tile, so no read can leave
//    it) with the non-temporal hint: the cache is streamed once, and on
//    MI355X the hint lifts a plain 4 KiB-tile gather from ~6.1 to ~6.9 TB/s.
//    A K load instruction reads 1 KiB of contiguous memory; a V load reads
//    four whole 256-byte token rows (D = 128).
//  * Scores, transposed.  S^T = K Q^T is D/32 MFMA f32_16x16x32_bf16 per
//    block with the K tile as the A operand (16 token rows) and the query
//    rows as the B operand.  The K cache stores each block as D/8 chunks of
//    [16 slots][8 elements], so the A fragment of lane l in k-step c -- 8
//    consecutive d of token l%16, chunk 4c + l/16 -- is exactly the 16 bytes
//    at offset 1024c + 16l of the tile; q uses the same assignment of d to
//    (k-step, k-group, element).  The result leaves lane (kg, n) with the
//    scores of query row n for tokens 4kg .. 4kg+3.
//  * Softmax.  The running maximum is moved only when some score of the block
//    exceeds it by more than 2^8 (a wavefront vote); then each row's block
//    max is reduced over its four lanes and the state is rescaled.
//    Otherwise probabilities are taken against the stale maximum (they stay
//    below 2^8, far inside fp32), so most blocks need neither the reduction
//    nor the rescale; the result is the same softmax.  Blocks that every row
//    sees whole take a path without any masking.
//  * P V, transposed, on MFMA.  O^T = V^T P^T is D/16 MFMA f32_16x16x16_bf16
//    per block and half (or D/16 f32_16x16x32_bf16 per pair of blocks staged
//    in LDS): the probabilities of lane (kg, n) are already the B fragment
//    (column n, k-group kg), and the A fragment of lane (kg, n) is 4 tokens
//    x 1 column of the V tile (of each block), picked out of the 16-byte row
//    pieces the lane loaded, or read transposed from LDS (pv_staged).  Each probability p is split into bf16 hi = p with the
//    low 16 bits cleared and lo = bf16(p - hi), and both halves go through
//    the MFMA, so P keeps about 16 significant bits (relative error below
//    2^-15) instead of bf16's 8.  The output of row n stays in the lanes of
//    row n: D/16 accumulators of 4 floats each, whatever the row count.
//  * Tokens a row must not see (past the context in the last block, or after
//    the row's own position for multi-token queries) are removed by
//    selection: score -inf, and V rows past the context set to zero, so
//    whatever those slots hold (NaN included) never reaches the result.
#pragma once

#include "pda_internal.h"

namespace pda {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short shortx4_t __attribute__((ext_vector_type(4)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// IEEE 754-2019 maximum of three values (NaN propagates; one instruction).
__device__ __forceinline__ float max3(float a, float b, float c) {
  return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}

// x * y rounded on its own: never fused with a following add.
__device__ __forceinline__ float mul_rounded(float x, float y) {
#pragma clang fp contract(off)
  return x * y;
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

// Two bf16 taken from the same half of two dwords, packed low-first:
// hi_half ? (a >> 16) | (b & 0xffff0000) : (a & 0xffff) | (b << 16).
__device__ __forceinline__ unsigned pack_halves(unsigned a, unsigned b, bool hi_half) {
  return __builtin_amdgcn_perm(b, a, hi_half ? 0x07060302u : 0x05040100u);
}

template <int D>
struct WaveAttention {
  static_assert(D == 64 || D == 128, "head_dim");
  static constexpr int NC = D / 32;               // score MFMA k-steps per block
  static constexpr int VT = D / 16;               // P.V MFMA output tiles (16 d each)
  static constexpr int kRowBytes = D * 2;         // one token row of a V tile
  static constexpr int kTileBytes = kBlockTokens * kRowBytes;
  static constexpr int kStagedRow = D + 16;       // elements per V row staged in LDS (32 bytes of padding)
  static constexpr float kNegInf = -__builtin_huge_valf();
  static constexpr float kFloor = -1e30f;         // running max of a row that has seen no token
  static constexpr float kRescaleSlack = 8.f;     // log2 of the largest unnormalised probability

  int lane, n, kg;
  int k_off, v_off;  // this lane's byte offsets in a K / V tile
  int tr_off;        // this lane's element offset in a V tile for transposed reads (pv_staged)
  bool tr_cols;      // o[t][i] holds output column 16t + 4kg + i (pv_staged) instead of d_of(i, t)
  int lim_off;       // this lane's query row sees tokens t < L - lim_off
  float scale_log2;
  bool bad;          // a block id outside the pool was met (never dereferenced)
  bf16x8_t qa[NC];
  floatx4_t o[VT];
  float m_run, l_run;

  __device__ __forceinline__ explicit WaveAttention(float scale_log2_) : scale_log2(scale_log2_), bad(false) {
    lane = threadIdx.x & (kWaveSize - 1);
    n = lane & 15;
    kg = lane >> 4;
    k_off = 16 * lane;
    v_off = 4 * kg * kRowBytes + 16 * (n % (D / 8));
    tr_off = (4 * kg + n / 4) * kStagedRow + 4 * (n % 4);
    tr_cols = false;
  }

  // The output element d of this lane's row held in accumulator t, register i.
  // D = 128: A row r of tile t is column 8r + t, and C row 4kg + i is A row
  // 4kg + i.  D = 64: lanes n and n + 8 load the same 8 columns, and A row r
  // of tile t is column 8 (r % 8) + t + 4 (r / 8).
  __device__ __forceinline__ int d_of(int i, int t) const {
    const int r = 4 * kg + i;
    return D == 128 ? 8 * r + t : 8 * (r & 7) + t + 4 * (r >> 3);
  }

  // Load this lane's query row (`q_row`: D bf16) and clear the state; the row
  // sees context tokens t < L - lim_off_.
  __device__ __forceinline__ void start(const uint16_t* q_row, int lim_off_) {
    bad = false;
    lim_off = lim_off_;
    const uint16_t* p = q_row + kg * 8;
#pragma unroll
    for (int c = 0; c < NC; ++c) qa[c] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(p + 32 * c));
#pragma unroll
    for (int t = 0; t < VT; ++t) o[t] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    m_run = kFloor;
    l_run = 0.f;
  }

  // Issue the K and V tile loads of one block (or, when !needed, loads through a
  // zero-length descriptor that the hardware drops without touching memory).
  __device__ __forceinline__ void load_tiles(uint4 (&kr)[NC], uint4 (&vr)[4], const char* kpool, const char* vpool,
                                             size_t block_bytes, int num_blocks, int phys, bool needed) {
    if ((unsigned)phys >= (unsigned)num_blocks) {  // contract violation: never read outside the pool
      bad = true;
      phys = 0;
    }
    const size_t off = (size_t)phys * block_bytes;
    const int bytes = needed ? kTileBytes : 0;
    const __amdgpu_buffer_rsrc_t rk = tile_rsrc(kpool + off, bytes);
    const __amdgpu_buffer_rsrc_t rv = tile_rsrc(vpool + off, bytes);
#pragma unroll
    for (int c = 0; c < NC; ++c) kr[c] = load_stream(rk, k_off + c * 1024);
#pragma unroll
    for (int e = 0; e < 4; ++e) vr[e] = load_stream(rv, v_off + e * kRowBytes);
  }

  // The dword of token row e of a V tile piece `v` that holds this lane's
  // column of output tile t (the column d_of gives for accumulator row 4kg+e).
  __device__ __forceinline__ unsigned col_dword(const uint4 (&v)[4], int e, int t) const {
    const int dw = t >> 1;
    if (D == 128) return dw == 0 ? v[e].x : dw == 1 ? v[e].y : dw == 2 ? v[e].z : v[e].w;
    const bool upper = n >= 8;  // D = 64: lanes n and n + 8 hold the same 8 columns
    return dw == 0 ? (upper ? v[e].z : v[e].x) : (upper ? v[e].w : v[e].y);
  }

  // Move the running max to cover `mx` (this lane's largest scaled score),
  // reduced over the row's four lanes, and rescale the state.
  __device__ __forceinline__ void rescale(float mx) {
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mn = fmaxf(m_run, mx);  // the same in the four lanes of the row
    const float al = exp2_fast(m_run - mn);
    m_run = mn;
    l_run *= al;
#pragma unroll
    for (int t = 0; t < VT; ++t) o[t] *= al;
  }

  // P^T of NB blocks as two bf16 B fragments per block: hi = p truncated,
  // lo = bf16(p - hi); word 2b + h holds tokens 4kg + 2h, 4kg + 2h + 1 of block b.
  template <int NB>
  struct PFrag {
    unsigned hw[2 * NB], lw[2 * NB];
  };

  // Fold the scores of NB consecutive blocks (NB = 1 or 2; logical tokens
  // tok0 .. tok0 + 16 NB - 1) into the softmax state and return their
  // probabilities.  `tail` (wave-uniform): some row may not see some of these
  // tokens (the context ends in them, or a multi-token row's own position
  // comes before them, or they lie at or past `t_stop`); only then is
  // anything masked.
  //
  // Lane (kg, n) gets row n, tokens 4kg + i of each block.  Each probability
  // is exp2(fl(s * scale) - max): the largest score of a row gets exactly 1,
  // so a one-token context returns its V row exactly.  A masked score is
  // -inf after scaling (so a zero scale masks too).
  template <int NB>
  __device__ __forceinline__ PFrag<NB> softmax(const uint4 (&kr)[NB][NC], int tok0, int L, bool tail,
                                               int t_stop = 0x7fffffff) {
    float sc[NB][4];
    scores<NB>(kr, sc);
    return probs<NB>(sc, tok0, L, tail, t_stop);
  }

  // The scaled scores of NB blocks: D/32 MFMAs per block, then the scaling.
  // The scaled scores are formed here, in the MFMAs' own basic block: the
  // compiler did not insert the wait states a VALU read of an MFMA result
  // needs when the first such read came after the tail branch of probs.
  // PRIO: the MFMAs issue at raised wave priority (as in pv_staged).
  template <int NB, bool PRIO = false>
  __device__ __forceinline__ void scores(const uint4 (&kr)[NB][NC], float (&sc)[NB][4]) const {
    floatx4_t acc[NB];
    if constexpr (PRIO) __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      acc[b] = floatx4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NC; ++c)
        acc[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kr[b][c]), qa[c], acc[b], 0, 0, 0);
    }
    if constexpr (PRIO) __builtin_amdgcn_s_setprio(0);
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) sc[b][i] = mul_rounded(acc[b][i], scale_log2);
  }

  // The masking, the running max and the probabilities of scaled scores.
  template <int NB>
  __device__ __forceinline__ PFrag<NB> probs(float (&sc)[NB][4], int tok0, int L, bool tail, int t_stop) {
    if (tail) {
      // An empty volatile asm keeps this a branch: as selects, the masking
      // would run on every block.
      asm volatile("");
      const int rel = min(L - lim_off, t_stop) - (tok0 + 4 * kg);  // this lane's first token at or past it is masked
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (kBlockTokens * b + i >= rel) sc[b][i] = kNegInf;
    }
    // IEEE maximum (v_maximum3_f32): unlike fmaxf it needs no quieting of
    // its inputs, which come from another basic block after the masking.
    float top = max3(sc[0][0], sc[0][1], max3(sc[0][2], sc[0][3], NB == 2 ? sc[1][0] : kNegInf));
    if constexpr (NB == 2) top = max3(top, max3(sc[1][1], sc[1][2], sc[1][3]), kNegInf);
    if (__builtin_amdgcn_ballot_w64(top > m_run + kRescaleSlack) != 0) rescale(top);  // wave-uniform
    float pr[NB][4];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) pr[b][i] = exp2_fast(sc[b][i] - m_run);
    float ls = (pr[0][0] + pr[0][1]) + (pr[0][2] + pr[0][3]);
    if constexpr (NB == 2) ls += (pr[1][0] + pr[1][1]) + (pr[1][2] + pr[1][3]);
    l_run += ls;
    PFrag<NB> f;
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const unsigned h0 = __float_as_uint(pr[b][2 * h]) & 0xffff0000u;
        const unsigned h1 = __float_as_uint(pr[b][2 * h + 1]) & 0xffff0000u;
        f.hw[2 * b + h] = pack_halves(h0, h1, true);
        typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
        const bf16x2_t l2 = {(__bf16)(pr[b][2 * h] - __uint_as_float(h0)),
                             (__bf16)(pr[b][2 * h + 1] - __uint_as_float(h1))};
        f.lw[2 * b + h] = __builtin_bit_cast(unsigned, l2);
      }
    return f;
  }

  // Zero the V rows at or past `l_vis` (no row of the chunk sees them), so
  // whatever those slots hold never meets a zero probability.
  __device__ __forceinline__ void mask_v(uint4 (&vr)[4], int tok0, int l_vis, bool tail) const {
    if (tail) {
      asm volatile("");  // a branch, as in softmax
      const int rel = l_vis - (tok0 + 4 * kg);  // this lane's rows from it on are zeroed
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (e >= rel) vr[e] = make_uint4(0u, 0u, 0u, 0u);
    }
  }

  // O^T += V^T P^T for one block whose V rows 4kg .. 4kg+3 this lane holds
  // (16 bytes of each): D/16 MFMA f32_16x16x16_bf16 per half of P, the A
  // fragment of tile t picked out of those row pieces.
  __device__ __forceinline__ void pv(const uint4 (&vr)[4], const PFrag<1>& f) {
    const shortx4_t bh = __builtin_bit_cast(shortx4_t, make_uint2(f.hw[0], f.hw[1]));
    const shortx4_t bl = __builtin_bit_cast(shortx4_t, make_uint2(f.lw[0], f.lw[1]));
#pragma unroll
    for (int t = 0; t < VT; ++t) {
      const bool hi_half = t & 1;
      const shortx4_t a = __builtin_bit_cast(
          shortx4_t, make_uint2(pack_halves(col_dword(vr, 0, t), col_dword(vr, 1, t), hi_half),
                                pack_halves(col_dword(vr, 2, t), col_dword(vr, 3, t), hi_half)));
      o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, bh, o[t], 0, 0, 0);
      o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, bl, o[t], 0, 0, 0);
    }
  }

  // The V^T A fragments of a pair of blocks whose V tiles (16 rows of D
  // bf16, kStagedRow elements apart) are in LDS at va and vb, read straight
  // from LDS through transposed reads (ds_read_b64_tr_b16): within each group
  // of 16 lanes, source lane s reads 4 consecutive elements at its own
  // address, and lane m receives element m % 4 of source lanes m / 4,
  // m / 4 + 4, m / 4 + 8, m / 4 + 12.  With source lane (kg, s) pointing at
  // row 4kg + s / 4, columns 16t + 4 (s % 4), lane (kg, m) receives
  // V[4kg + j][16t + m], j = 0..3: tokens 4kg .. 4kg+3, as its
  // probabilities, and column 16t + m, so the accumulators take the tr_cols
  // assignment.  No v_perm is needed.  The caller reads them before the
  // pair's softmax, so that the LDS latency overlaps it.
  __device__ __forceinline__ void v_frags(const uint16_t* va, const uint16_t* vb, uint4 (&aw)[VT]) const {
    typedef short v4s_t __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) v4s_t lds_v4s_t;
#pragma unroll
    for (int t = 0; t < VT; ++t) {
      const uint2 x = __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                                    (lds_v4s_t*)(va + tr_off + 16 * t)));
      const uint2 y = __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                                    (lds_v4s_t*)(vb + tr_off + 16 * t)));
      aw[t] = make_uint4(x.x, x.y, y.x, y.y);
    }
  }

  // O^T += V^T P^T for a staged pair (fragments from v_frags), with D/16
  // MFMA f32_16x16x32_bf16 per half of P.  In a tail pair, fragment elements
  // of tokens at or past l_vis are zeroed first.  PRIO: the wavefront issues
  // these MFMAs at raised priority (for workgroups of 8 wavefronts, whose
  // pairs on a SIMD fold the same steps; with the score MFMAs raised too,
  // chunked prefill and long CoT with 64 new tokens ran 5% faster on MI355X,
  // while workgroups of 4 gained nothing and lost 4.6% with 16 new tokens).
  template <bool PRIO = false>
  __device__ __forceinline__ void pv_staged(uint4 (&aw)[VT], const PFrag<2>& f, bool tail, int tok0, int l_vis) {
    if (tail) {
      asm volatile("");  // a branch, as in softmax
      const int rel = l_vis - (tok0 + 4 * kg);  // this lane's tokens below it are kept
      unsigned mw[4];
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int t0 = kBlockTokens * b + 2 * h;
          mw[2 * b + h] = (t0 < rel ? 0x0000ffffu : 0u) | (t0 + 1 < rel ? 0xffff0000u : 0u);
        }
#pragma unroll
      for (int t = 0; t < VT; ++t) aw[t] = make_uint4(aw[t].x & mw[0], aw[t].y & mw[1], aw[t].z & mw[2], aw[t].w & mw[3]);
    }
    const bf16x8_t bh = __builtin_bit_cast(bf16x8_t, make_uint4(f.hw[0], f.hw[1], f.hw[2], f.hw[3]));
    const bf16x8_t bl = __builtin_bit_cast(bf16x8_t, make_uint4(f.lw[0], f.lw[1], f.lw[2], f.lw[3]));
    if constexpr (PRIO) __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int t = 0; t < VT; ++t) {
      const bf16x8_t a = __builtin_bit_cast(bf16x8_t, aw[t]);
      o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bh, o[t], 0, 0, 0);
      o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bl, o[t], 0, 0, 0);
    }
    if constexpr (PRIO) __builtin_amdgcn_s_setprio(0);
  }

  // Fold one block (logical tokens tok0 .. tok0+15) into the state.  `L` is
  // the context length, `l_first` the limit of the chunk's first row (every
  // row sees tokens below it) and `l_vis` the limit of its last row (no row
  // sees a token at or above it).
  __device__ __forceinline__ void process(const uint4 (&kr)[NC], uint4 (&vr)[4], int tok0, int L, int l_first,
                                          int l_vis) {
    uint4 k1[1][NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) k1[0][c] = kr[c];
    const bool tail = tok0 + kBlockTokens > l_first;  // wave-uniform
    const PFrag<1> f = softmax<1>(k1, tok0, L, tail);
    mask_v(vr, tok0, l_vis, tail);
    pv(vr, f);
  }

  // Stream blocks [j0, j1) of one sequence: block ids in `table_row`, tiles of
  // this KV head at kpool/vpool + id * block_bytes; L, l_first, l_vis as in
  // process().
  //
  // Two register buffers: the tiles of block i+1 are in flight while block i
  // is computed.  Every load is unconditional, so the compiler counts
  // outstanding loads exactly and waits only for the tiles it is about to
  // use; the scheduling barriers keep each prefetch ahead of the first use of
  // the current tiles.  Past the end of the run the prefetch gets a
  // zero-length descriptor.  Block ids come 64 at a time, one per lane, and
  // are read with readlane, so no tile load waits on a scalar load.
  __device__ __forceinline__ void run(const int32_t* table_row, int j0, int j1, int L, int l_first, int l_vis,
                                      const char* kpool, const char* vpool, size_t block_bytes, int num_blocks) {
    const int cnt = j1 - j0;
    uint4 k0[NC], v0[4], k1[NC], v1[4];
    for (int c0 = 0; c0 < cnt; c0 += kWaveSize) {
      const int cn = min(kWaveSize, cnt - c0);
      const int jc = j0 + c0;
      const int ids = lane < cn ? table_row[jc + lane] : 0;
      auto id = [&](int i) { return __builtin_amdgcn_readlane(ids, i); };
      load_tiles(k0, v0, kpool, vpool, block_bytes, num_blocks, id(0), true);
      for (int i = 0; i < cn; i += 2) {
        load_tiles(k1, v1, kpool, vpool, block_bytes, num_blocks, id(min(i + 1, cn - 1)), i + 1 < cn);
        __builtin_amdgcn_sched_barrier(0);
        process(k0, v0, (jc + i) * kBlockTokens, L, l_first, l_vis);
        if (i + 1 >= cn) break;
        load_tiles(k0, v0, kpool, vpool, block_bytes, num_blocks, id(min(i + 2, cn - 1)), i + 2 < cn);
        __builtin_amdgcn_sched_barrier(0);
        process(k1, v1, (jc + i + 1) * kBlockTokens, L, l_first, l_vis);
      }
    }
  }

  // Sum each row's denominator over its four lanes (a fixed butterfly, so the
  // four lanes hold the same bits).  The running max is already the same in
  // the four lanes, and the output of row n is complete in them.
  __device__ __forceinline__ void finish() {
    l_run += __shfl_xor(l_run, 16);
    l_run += __shfl_xor(l_run, 32);
  }
};

}  // namespace pda
