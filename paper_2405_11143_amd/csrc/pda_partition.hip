// Pass 1: one workgroup per work item, taken in the order pda_order.hip
// computed (largest first, placed for the XCDs), or in natural order when
// every item runs at once.  Two kinds of items share the launch:
//
// Regular items: (partition of a context, sequence, KV head, group of up to
// 4 chunks of new query tokens, up to 8 when there are more than 4, up to 16
// when there are more than 8).  A chunk holds up to 16 / G consecutive new
// tokens of the sequence, so its query rows (token-major, then the G heads of
// the KV head) fill one 16-row MFMA tile; a decode step has one token, i.e.
// one chunk of G rows.  New token i of a sequence with n new tokens and
// context length L sits at position L - n + i and sees tokens
// t < L - n + 1 + i.  The 4 wavefronts take the item's chunks first and
// slices of its blocks second (1 chunk: 4 contiguous runs; 2: every other
// step of 2 blocks each; 3-4: every block; 5-8, the wide variant: chunks w
// and w + 4 on wavefront w, every block; 9-16, the wide variant on 8
// wavefronts: chunks w and w + 8), so the chunks of one item read each tile
// on one compute unit.  Each chunk keeps its own causal range and
// partition count.  With shared-prefix groups, a sequence's regular items
// cover only the tokens after its group's prefix.
//
// Prefix items: (shared-prefix group, prefix partition, row group, KV head).
// All members of a group read the same prefix blocks (parallel sampling,
// Section 3.2), so the prefix is attended once for all members x new tokens x
// G heads of a row group (64 / (n G) members, up to 64 query rows; larger
// groups take several row groups, each reading the prefix once; a row whose
// position lies inside the prefix sees only the prefix tokens before it):
// the 4 wavefronts take 16-row tiles first and slices of blocks second, as
// above, and every block's tiles reach the compute unit once per row group.
//
// With one tile, each wavefront streams its run of 16-token blocks with
// WaveAttention (pda_wave.h), tiles straight into registers.  With several
// tiles, the workgroup stages every block's K and V tiles through LDS once
// (2 blocks per step, two steps in flight) and each wavefront folds them
// from there for its own rows, a pair of blocks at a time.  The states of
// the wavefronts that share a row are merged through LDS in a fixed order.
// A regular item with no prefix that sees a single partition writes its
// final output rows; every other item leaves a partial softmax state (max,
// denominator, unnormalised output) for the merge pass.  Nothing depends on physical block ids or on timing, so results
// are bit-for-bit reproducible and independent of block placement.
#include "pda_wave.h"

namespace pda {
namespace {

constexpr int kRows = 16;           // rows of one wavefront (one MFMA tile)

template <int D, int NW>
struct PassShared {
  float o[NW][kRows][D];
  float m[NW][kRows];
  float l[NW][kRows];
  float sc[NW][kRows];    // per wavefront and row: 2^(m - M), M the row's max over its slices
  float mx[NW][kRows];    // per tile and row: M
  float lsum[NW][kRows];  // per tile and row: sum of sc * l over the slices
  int bad[NW];
};

// Tile staging for items with several 16-row tiles: every step brings SB
// consecutive blocks' K and V tiles into LDS, loaded once by the whole
// workgroup, and every wavefront reads its MFMA fragments from there.  Three
// buffers: one step is folded while the loads of the next two are in flight
// (in registers, then written to LDS).  Block ids come through an LDS window.
constexpr int kIdWindow = 256;

template <int D, int SB, int NW>
struct Staging {
  static constexpr int kStepBlocks = SB;
  static constexpr int TC = WaveAttention<D>::kTileBytes / 16;       // 16-byte pieces per tile
  static constexpr int kLoads = SB * 2 * TC / (NW * kWaveSize);  // per thread and step
  static constexpr int kRowPieces = D / 8;                            // 16-byte pieces per V row
  // A block is its K tile as loaded, then its V tile with 32 bytes of padding
  // after every row: a transposed V read takes 32 bytes from each of 4 rows
  // per group of 16 lanes, and with the padding those rows start 8 banks
  // apart, so the 4 pieces fall on disjoint banks (unpadded the staged step
  // ran 10% slower; 16 bytes of padding, which overlaps neighbouring rows'
  // banks by half, ran 0.5-1.3% slower than 32 on MI355X).
  static constexpr int kBlockPieces = TC + kBlockTokens * (kRowPieces + 2);
  uint4 buf[3][SB][kBlockPieces];
  int ids[kIdWindow];
};

// Which paths a launch compiles.  A launch whose items all have one tile
// (every decode step without shared-prefix groups) compiles the register
// path only (138 VGPRs at D = 128, 33 KiB of LDS); with up to 4 query chunks
// per item both paths are compiled (167 VGPRs, 50.5 KiB); with more, the
// wide variant also folds two tiles per wavefront (243 VGPRs, 2
// workgroups per compute unit), and beyond 8 chunks its 8-wavefront form
// does (227 VGPRs, 67 KiB, one workgroup per compute unit: each staged step
// then serves 16 tiles, half the staging and barriers per tile of 8).
// Staging takes 2 blocks per step, so three
// staging buffers (49.5 KiB at D = 128) still leave room for 3 workgroups
// per compute unit; 4 blocks per step at 2 workgroups per compute unit
// measured slower on MI355X.
constexpr int kModeRegister = 1, kModeMixed = 3, kModeWide = 7, kModeWide16 = 15;
constexpr int kStepBlocks = 2;

// Wavefronts per workgroup: 8 in the variant for items of more than 8 query
// chunks (two tiles each, 16 chunks sharing every staged step), 4 otherwise.
constexpr int waves_of(int mode) { return mode == kModeWide16 ? 2 * kWaves : kWaves; }
constexpr bool wide_mode(int mode) { return mode == kModeWide || mode == kModeWide16; }

template <int D, int MODE>
union PassLds {
  PassShared<D, waves_of(MODE)> sh;                // the epilogue
  Staging<D, kStepBlocks, waves_of(MODE)> st;      // the staged main loop (never live at the same time)
};

template <int D>
union PassLds<D, kModeRegister> {  // no staging in the register-only variant
  PassShared<D, kWaves> sh;
};

// Publish a finished wavefront's state: rows n < rows of the tile.
template <int D, int NW>
__device__ __forceinline__ void publish(PassShared<D, NW>& sh, const WaveAttention<D>& wave, int w, int lane,
                                        int rows) {
  const int n = lane & 15;
  if (n < rows) {
    if (wave.tr_cols) {  // o[t][i] = column 16t + 4kg + i
#pragma unroll
      for (int t = 0; t < WaveAttention<D>::VT; ++t)
        *reinterpret_cast<float4*>(&sh.o[w][n][16 * t + 4 * wave.kg]) =
            make_float4(wave.o[t][0], wave.o[t][1], wave.o[t][2], wave.o[t][3]);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d0 = wave.d_of(i, 0);  // D = 128: 8 consecutive columns; D = 64: 4
        *reinterpret_cast<float4*>(&sh.o[w][n][d0]) =
            make_float4(wave.o[0][i], wave.o[1][i], wave.o[2][i], wave.o[3][i]);
        if constexpr (D == 128)
          *reinterpret_cast<float4*>(&sh.o[w][n][d0 + 4]) =
              make_float4(wave.o[4][i], wave.o[5][i], wave.o[6][i], wave.o[7][i]);
      }
    }
    if (lane < 16) {
      sh.m[w][n] = wave.m_run;
      sh.l[w][n] = wave.l_run;
    }
  }
  if (lane == 0) sh.bad[w] = wave.bad ? 1 : 0;
}

// The weights that merge the slices of each tile, once per row: for tile t
// (wavefronts t, t + ntile, ... : `slices` of them) and row h, the max M of
// their running maxima, each one's scale 2^(m - M) (0 for a wavefront that
// saw no token of the row) and the scaled sum of their denominators, all in
// a fixed order.  Rows past a tile's last one hold values nobody reads.
// Ends with a barrier.
template <int D, int NW>
__device__ __forceinline__ void row_weights(PassShared<D, NW>& sh, int ntile, int slices) {
  const int tid = threadIdx.x;
  if (tid < ntile * kRows) {
    const int t = tid / kRows;
    const int h = tid % kRows;
    float M = WaveAttention<D>::kFloor;
    for (int x = 0; x < slices; ++x) M = fmaxf(M, sh.m[t + x * ntile][h]);
    float lsum = 0.f;
    for (int x = 0; x < slices; ++x) {
      const int w = t + x * ntile;
      const float sc = exp2_fast(sh.m[w][h] - M);
      sh.sc[w][h] = sc;
      lsum = fmaf(sc, sh.l[w][h], lsum);
    }
    sh.mx[t][h] = M;
    sh.lsum[t][h] = lsum;
  }
  __syncthreads();
}

// One merged output element of tile t, row h, column d (row_weights first).
template <int D, int NW>
__device__ __forceinline__ float combine(const PassShared<D, NW>& sh, int t, int ntile, int slices, int h, int d) {
  float acc = 0.f;
  for (int x = 0; x < slices; ++x) {
    const int w = t + x * ntile;
    acc = fmaf(sh.sc[w][h], sh.o[w][h][d], acc);
  }
  return acc;
}

// The partial state of one row and partition: 4 output columns d0 .. d0+3,
// and with the first of them the max and the denominator.  Plain (cached)
// stores: the merge pass reads them right after.
__device__ __forceinline__ void store_partial4(const StepArgs& a, size_t slot, int d0, int D, const float (&acc)[4],
                                               float M, float lsum) {
  *reinterpret_cast<f32x4_t*>(a.part_o + slot * D + d0) = f32x4_t{acc[0], acc[1], acc[2], acc[3]};
  if (d0 == 0) {
    a.part_m[slot] = M;
    a.part_l[slot] = lsum;
  }
}

// One final output row's columns d0 .. d0+3: acc / lsum, or acc itself (0,
// or NaN) for a row that sees nothing.
__device__ __forceinline__ void store_final4(float* p, const float (&acc)[4], float lsum) {
  const bool pos = lsum > 0.f;
  store_nt4(p, pos ? acc[0] / lsum : acc[0], pos ? acc[1] / lsum : acc[1], pos ? acc[2] / lsum : acc[2],
            pos ? acc[3] / lsum : acc[3]);
}

// Stream blocks [J0, J1) of one sequence through LDS, a step of 2 blocks at a
// time.  All threads of the workgroup call this.  Wavefront (tile, slice)
// folds the steps slice, slice + slices, ... of each window into its state,
// both blocks of a step as one pair (every fold is a pair, so the output
// accumulators stay put), and only blocks below its own end `j_stop` (its
// query chunk's causal range); an inactive wavefront only helps to load.
// With NT = 2 the wavefront also folds a second, later chunk into `wave_b`
// (blocks below j_stop_b, which is 0 when it has none) from the same K and V
// fragments.
template <int D, int SB, int NT, int NW>
__device__ void run_staged(WaveAttention<D>& wave, WaveAttention<D>& wave_b, Staging<D, SB, NW>& st,
                           const int32_t* table_row, int J0, int J1, int j_stop, int j_stop_b, bool active, int slice,
                           int slices, int L, int l_first, int l_vis, int l_first_b, int l_vis_b, const char* kpool,
                           const char* vpool, size_t block_bytes, int num_blocks) {
  using WA = WaveAttention<D>;
  static_assert(SB == 2, "a step is one pair of blocks");
  static_assert(Staging<D, SB, NW>::TC % kWaveSize == 0, "a wavefront's loads stay within one tile");
  wave.tr_cols = true;  // every fold here goes through pv_staged
  wave_b.tr_cols = true;
  constexpr int TC = Staging<D, SB, NW>::TC;
  constexpr int NL = Staging<D, SB, NW>::kLoads;
  const int tid = threadIdx.x;
  bool bad = false;
  // Two steps' loads are in flight in two register sets while a third
  // step is folded from LDS (three buffers); in the wide variants' folds,
  // three steps in three register sets (their registers allow it at 2
  // wavefronts per SIMD; on MI355X 0.2-0.8% faster on every wide step).
  uint4 ra[NL], rb[NL], rc[NL];
  constexpr bool kThree = NW == 2 * kWaves || (NW == kWaves && NT == 2);
  // Load k of a thread takes piece ci = k * 256 + tid of the step, in
  // [block][K or V][piece] order.  A tile is a multiple of 64 pieces, so the
  // 64 lanes of a wavefront share the block and the K or V side of each load:
  // both are taken from the wavefront's first piece, and the block ids go
  // through scalar registers, so every load has one buffer descriptor per
  // wavefront (a per-lane one costs a loop over the distinct values).
  const int wbase = __builtin_amdgcn_readfirstlane(tid & ~(kWaveSize - 1));
  const int lane_piece = tid & (kWaveSize - 1);
  // issue the loads of step `step` of the window starting at block jw
  auto issue = [&](uint4(&r)[NL], int jw, int jwe, int step) {
    int phys[SB], bytes[SB];  // (readfirstlane keeps them in scalar registers)
#pragma unroll
    for (int s = 0; s < SB; ++s) {
      const int j = jw + step * SB + s;
      const bool valid = j < jwe;
      int id = __builtin_amdgcn_readfirstlane(valid ? st.ids[j - jw] : 0);
      if ((unsigned)id >= (unsigned)num_blocks) {  // contract violation: never read outside the pool
        bad |= valid;
        id = 0;
      }
      phys[s] = id;
      bytes[s] = __builtin_amdgcn_readfirstlane(valid ? WA::kTileBytes : 0);
    }
#pragma unroll
    for (int k = 0; k < NL; ++k) {
      const int cb = k * NW * kWaveSize + wbase;  // the wavefront's first piece
      const int blk = cb / (2 * TC);
      const char* pool = ((cb / TC) & 1) ? vpool : kpool;
      r[k] = load_stream(tile_rsrc(pool + (size_t)(blk == 0 ? phys[0] : phys[1]) * block_bytes,
                                   __builtin_amdgcn_readfirstlane(blk == 0 ? bytes[0] : bytes[1])),
                         (cb % TC + lane_piece) * 16);
    }
  };
  // where each of this thread's loads goes in a step's buffer
  int dst[NL];
#pragma unroll
  for (int k = 0; k < NL; ++k) {
    const int ci = k * NW * kWaveSize + tid;  // [block][K or V][piece]
    const int pc = ci % TC;
    constexpr int RP = Staging<D, SB, NW>::kRowPieces;
    dst[k] = ci / (2 * TC) * Staging<D, SB, NW>::kBlockPieces +
             (((ci / TC) & 1) ? TC + pc / RP * (RP + 2) + pc % RP : pc);
  }
  auto commit = [&](const uint4(&r)[NL], int buf) {
#pragma unroll
    for (int k = 0; k < NL; ++k) (&st.buf[buf][0][0])[dst[k]] = r[k];
  };
  // fold step `step` (in buffer buf) if it is this wavefront's
  auto fold_step = [&](int jw, int jwe, int step, int buf) {
    if (!active || step % slices != slice) return;  // wave-uniform
    // Both blocks of the step as one pair.  When only the first is a chunk's
    // (the run or its causal range ends there), the second is masked whole
    // through t_stop (its slot in LDS holds zeros or another range's tiles).
    const int j0 = jw + step * SB;
    const int j_lim = min(jwe, j_stop);
    const int j_lim_b = NT == 2 ? min(jwe, j_stop_b) : 0;
    const bool fold_a = j0 < j_lim;
    const bool fold_b = NT == 2 && j0 < j_lim_b;
    if (!fold_a && !fold_b) return;
    const int tok0 = j0 * kBlockTokens;
    uint4 kr[2][WA::NC];
#pragma unroll
    for (int k = 0; k < 2; ++k)
#pragma unroll
      for (int c = 0; c < WA::NC; ++c) kr[k][c] = st.buf[buf][k][(c * 1024) / 16 + wave.lane];
    uint4 aw[WA::VT];
    wave.v_frags(reinterpret_cast<const uint16_t*>(st.buf[buf][0] + TC),
                 reinterpret_cast<const uint16_t*>(st.buf[buf][1] + TC), aw);
    if constexpr (NT == 2) {
      // Both chunks' score MFMAs first, back to back (a chunk that does not
      // fold this step discards its scores), so that those of the earlier
      // chunk run under the later chunk's softmax.  The later chunk folds
      // first: pv_staged zeroes (in aw) the V rows its last row does not
      // see, which no row of the earlier chunk sees either; the earlier
      // chunk's rows give the rows between them probability 0.
      float sc_b[2][4], sc_a[2][4];
      wave_b.template scores<2, NW == 2 * kWaves>(kr, sc_b);
      wave.template scores<2, NW == 2 * kWaves>(kr, sc_a);
      if (fold_b) {
        const int t_stop = j_lim_b * kBlockTokens;
        const bool tail = tok0 + 2 * kBlockTokens > min(l_first_b, t_stop);  // wave-uniform
        const auto f = wave_b.template probs<2>(sc_b, tok0, L, tail, t_stop);
        wave_b.template pv_staged<NW == 2 * kWaves>(aw, f, tail, tok0, min(l_vis_b, t_stop));
      }
      if (fold_a) {
        const int t_stop = j_lim * kBlockTokens;
        const bool tail = tok0 + 2 * kBlockTokens > min(l_first, t_stop);  // wave-uniform
        const auto f = wave.template probs<2>(sc_a, tok0, L, tail, t_stop);
        wave.template pv_staged<NW == 2 * kWaves>(aw, f, tail, tok0, min(l_vis, t_stop));
      }
    } else {
      const int t_stop = j_lim * kBlockTokens;
      const bool tail = tok0 + 2 * kBlockTokens > min(l_first, t_stop);  // wave-uniform
      const auto f = wave.template softmax<2>(kr, tok0, L, tail, t_stop);
      wave.template pv_staged<NW == 2 * kWaves>(aw, f, tail, tok0, min(l_vis, t_stop));
    }
  };
  for (int jw = J0; jw < J1; jw += kIdWindow) {
    const int jwe = min(J1, jw + kIdWindow);
    for (int j = jw + tid; j < jwe; j += NW * kWaveSize) st.ids[j - jw] = table_row[j];
    __syncthreads();
    const int nsteps = (jwe - jw + SB - 1) / SB;
    if constexpr (!kThree) {
      issue(ra, jw, jwe, 0);
      if (nsteps > 1) issue(rb, jw, jwe, 1);
      commit(ra, 0);
      __syncthreads();
      if (nsteps > 2) issue(ra, jw, jwe, 2);
      // Step s sits in buffer s % 3; before the barrier that ends step s, step
      // s + 1 moves from its registers into buffer (s + 1) % 3 (last read in
      // step s - 2), and after it the freed registers take step s + 3.
      // Unrolled by two so that the register sets stay static.
      for (int step = 0, buf = 0; step < nsteps; step += 2) {
        fold_step(jw, jwe, step, buf);
        buf = buf == 2 ? 0 : buf + 1;
        if (step + 1 < nsteps) commit(rb, buf);
        __syncthreads();
        if (step + 3 < nsteps) issue(rb, jw, jwe, step + 3);
        if (step + 1 >= nsteps) break;
        fold_step(jw, jwe, step + 1, buf);
        buf = buf == 2 ? 0 : buf + 1;
        if (step + 2 < nsteps) commit(ra, buf);
        __syncthreads();
        if (step + 4 < nsteps) issue(ra, jw, jwe, step + 4);
      }
    } else {
      // Three register sets: while step s is folded, steps s + 1 .. s + 3 are
      // in flight; the buffers are as above.  Unrolled by three.
      issue(ra, jw, jwe, 0);
      if (nsteps > 1) issue(rb, jw, jwe, 1);
      if (nsteps > 2) issue(rc, jw, jwe, 2);
      commit(ra, 0);
      __syncthreads();
      if (nsteps > 3) issue(ra, jw, jwe, 3);
      for (int step = 0, buf = 0; step < nsteps; step += 3) {
        fold_step(jw, jwe, step, buf);
        buf = buf == 2 ? 0 : buf + 1;
        if (step + 1 < nsteps) commit(rb, buf);
        __syncthreads();
        if (step + 4 < nsteps) issue(rb, jw, jwe, step + 4);
        if (step + 1 >= nsteps) break;
        fold_step(jw, jwe, step + 1, buf);
        buf = buf == 2 ? 0 : buf + 1;
        if (step + 2 < nsteps) commit(rc, buf);
        __syncthreads();
        if (step + 5 < nsteps) issue(rc, jw, jwe, step + 5);
        if (step + 2 >= nsteps) break;
        fold_step(jw, jwe, step + 2, buf);
        buf = buf == 2 ? 0 : buf + 1;
        if (step + 3 < nsteps) commit(ra, buf);
        __syncthreads();
        if (step + 6 < nsteps) issue(ra, jw, jwe, step + 6);
      }
    }
  }
  wave.bad |= __builtin_amdgcn_ballot_w64(bad) != 0;
  wave_b.bad |= wave.bad;
  __syncthreads();  // the staging area is reused by the epilogue
}

// The step's KV append folded into pass 1 (one new token per sequence, no
// shared-prefix groups): the wavefront whose run of blocks holds position t
// = L - 1 of (sequence b, KV head g) stores the new token's K and V rows
// there, and waits for the stores to complete, before it loads any tile.  No
// other wavefront or item reads that block (the last of the sequence's own
// context), and the wavefront's later loads of it miss its compute unit's
// L1 (stores do not allocate there), so they see the new rows.  A block id
// outside the pool is skipped, as the separate append does.
template <int D>
__device__ __forceinline__ void store_new_token(const StepArgs& a, int b, int g, int t, const int32_t* table_row,
                                                int lane) {
  constexpr int CPR = D / 8;  // 16-byte pieces per row
  const int phys = table_row[t / kBlockTokens];
  if ((unsigned)phys < (unsigned)a.num_blocks && lane < 2 * CPR) {
    const int c = lane % CPR;
    const size_t src = ((size_t)b * a.num_kv_heads + g) * CPR + c;
    const size_t tile = (size_t)phys * a.num_kv_heads + g;
    const int o = t % kBlockTokens;
    if (lane < CPR)
      reinterpret_cast<uint4*>(a.k_store)[(tile * CPR + c) * kBlockTokens + o] =
          reinterpret_cast<const uint4*>(a.k_new)[src];
    else
      reinterpret_cast<uint4*>(a.v_store)[(tile * kBlockTokens + o) * CPR + c] =
          reinterpret_cast<const uint4*>(a.v_new)[src];
  }
  __builtin_amdgcn_s_waitcnt(0);  // every memory operation of the wavefront has completed
}

template <int D, int MODE>
__device__ void regular_item(const StepArgs& a, PassLds<D, MODE>& lds, int item) {
  constexpr int NW = waves_of(MODE);
  PassShared<D, NW>& sh = lds.sh;
  using WA = WaveAttention<D>;
  const int Hq = a.num_q_heads;
  const int G = a.group;
  const int HC = a.num_kv_heads * a.num_chunk_groups;
  const int gc = item % HC;  // item = (p * B + b) * HC + g * NCG + chunk group
  const int b = (item / HC) % a.num_seqs;
  const int p = item / (HC * a.num_seqs);
  const int g = gc / a.num_chunk_groups;
  const int cg = gc % a.num_chunk_groups;
  const int nq = a.num_query_tokens;
  const int CPG = a.chunks_per_group;
  // query chunks (16-row tiles) of the item: always one in the register-only variant
  const int nchunk = MODE == kModeRegister ? 1 : min(CPG, a.num_query_chunks - cg * CPG);
  // more than 4 (wide variant only): wavefront w folds chunks w and, when it
  // exists, w + 4, and the epilogue takes the two sets of tiles in turn
  const bool two = wide_mode(MODE) && nchunk > NW;
  const int ntile = two ? NW : nchunk;  // tiles of the first (or only) set
  const int slices = NW / ntile;        // slices of blocks per tile
  const int tid = threadIdx.x;
  const int lane = tid & (kWaveSize - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int tile = w % ntile;
  const int slice = w / ntile;

  int L = a.lens[b];
  L = L < 0 ? 0 : (L > a.max_context_len ? a.max_context_len : L);
  const int Tp = a.partition_tokens;
  const int t0_all = seq_prefix_len(a, b);  // tokens before it belong to the group's prefix items
  // Per chunk c: its tokens [i0, i0 + nv), the token limit of its last row
  // (l_vis) and the partitions of its own tokens after the prefix.
  auto chunk_of = [&](int t) { return cg * CPG + t; };
  auto parts_of = [&](int c) {
    const int lv = chunk_visible(a, L, c);
    const int t0 = min(t0_all, max(lv, 0));
    return lv > 0 ? (lv - t0 + Tp - 1) / Tp : 0;
  };
  int nparts_max = 0;
  for (int t = 0; t < nchunk; ++t) nparts_max = max(nparts_max, parts_of(chunk_of(t)));
  if (p == 0) {  // chunks that see nothing (L == 0, or new tokens before the context): zero rows
    for (int t = 0; t < nchunk; ++t) {
      const int c = chunk_of(t);
      if (chunk_visible(a, L, c) > 0) continue;
      const int i0 = c * a.query_chunk;
      const int rows = min(a.query_chunk, nq - i0) * G;
      for (int i = tid; i < rows * D; i += NW * kWaveSize) {
        const int r = i / D;
        a.out[(((size_t)b * nq + i0 + r / G) * Hq + (size_t)g * G + r % G) * D + i % D] = 0.f;
      }
    }
  }
  if (p >= nparts_max) return;

  const char* kpool = reinterpret_cast<const char*>(a.k) + (size_t)g * WA::kTileBytes;
  const char* vpool = reinterpret_cast<const char*>(a.v) + (size_t)g * WA::kTileBytes;
  const int32_t* table_row = a.table + (size_t)b * a.max_blocks_per_seq;
  const size_t block_bytes = (size_t)a.num_kv_heads * WA::kTileBytes;
  // The partition's first block: that of the item's last chunk.  With a
  // shared prefix, every chunk with tokens after it starts its own range at
  // the prefix's end, as the last chunk does; a chunk whose rows see nothing
  // past the prefix has no own partitions and folds nothing.
  const int j_begin = (min(t0_all, max(chunk_visible(a, L, chunk_of(nchunk - 1)), 0)) + p * Tp) / kBlockTokens;
  auto block_end = [&](int lv, int parts) {  // end block of this partition for a chunk limit lv
    const int t0 = min(t0_all, max(lv, 0));
    return p < parts ? (min(lv, t0 + (p + 1) * Tp) + kBlockTokens - 1) / kBlockTokens : 0;
  };

  // One chunk's rows in a wavefront: lane row n repeats real rows past the
  // chunk's last one.
  struct ChunkRows {
    int c, rows, l_vis, l_first, nparts;
  };
  auto setup = [&](WA& wv, int c) {
    const int i0 = c * a.query_chunk;
    const int nv = min(a.query_chunk, nq - i0);
    ChunkRows cr{c, nv * G, chunk_visible(a, L, c), 0, parts_of(c)};
    cr.l_first = cr.l_vis - nv + 1;
    const int r = (lane & 15) % cr.rows;
    const int qi = i0 + r / G;
    wv.start(a.q + (((size_t)b * nq + qi) * Hq + (size_t)g * G + r % G) * D, nq - 1 - qi);
    return cr;
  };

  // Publish the wavefronts' states of the tiles [t_first, t_first + nt)
  // (wavefront w holds tile t_first + w % nt; `publishes` false: it holds
  // none of them), merge the slices of each in a fixed order and store
  // final rows or partial states.
  auto epilogue = [&](const WA& wv, int rows, bool publishes, int t_first, int nt, int sl, int& any_bad, bool first) {
    if (publishes) publish(sh, wv, w, lane, rows);
    __syncthreads();
    row_weights(sh, nt, sl);
    if (first) {
      any_bad = 0;
#pragma unroll
      for (int x = 0; x < NW; ++x) any_bad |= sh.bad[x];
    }
    for (int t = 0; t < nt; ++t) {
      const int ct = chunk_of(t_first + t);
      const int ct_parts = parts_of(ct);
      if (p >= ct_parts) continue;  // the chunk sees nothing in this partition
      const int ci0 = ct * a.query_chunk;
      const int crows = min(a.query_chunk, nq - ci0) * G;
      const bool single = ct_parts == 1 && min(t0_all, chunk_visible(a, L, ct)) == 0;
      for (int idx = tid; idx < crows * (D / 4); idx += NW * kWaveSize) {  // 4 columns per thread
        const int h = idx / (D / 4);
        const int d0 = 4 * (idx % (D / 4));
        float acc[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[e] = any_bad ? __builtin_nanf("") : combine(sh, t, nt, sl, h, d0 + e);
        const size_t row = ((size_t)b * nq + ci0 + h / G) * Hq + (size_t)g * G + h % G;
        if (single)
          store_final4(a.out + row * D + d0, acc, sh.lsum[t][h]);
        else
          store_partial4(a, row * a.slots_per_row + a.prefix_partitions + p, d0, D, acc, sh.mx[t][h], sh.lsum[t][h]);
      }
    }
  };

  WA wave(a.scale_log2);
  const ChunkRows ca = setup(wave, chunk_of(tile));
  if (MODE == kModeRegister && ntile != 1) return;  // not this launch's kind (never: the host picks the mode)
  int any_bad = 0;
  if (ntile == 1) {  // one tile: the 4 wavefronts split the blocks, tiles into registers
    const int j_end = block_end(ca.l_vis, ca.nparts);
    const int per_slice = (j_end - j_begin + NW - 1) / NW;
    const int wj0 = min(j_end, j_begin + w * per_slice);
    const int wj1 = min(j_end, wj0 + per_slice);
    if (a.k_new && L > 0 && wj0 <= (L - 1) / kBlockTokens && (L - 1) / kBlockTokens < wj1)  // wavefront-uniform
      store_new_token<D>(a, b, g, L - 1, table_row, lane);
    wave.run(table_row, wj0, wj1, L, ca.l_first, max(ca.l_vis, 0), kpool, vpool, block_bytes, a.num_blocks);
  } else if constexpr (MODE != kModeRegister) {  // several tiles: every block staged once through LDS for all of them
    int J1 = j_begin;
    for (int t = 0; t < nchunk; ++t) {
      const int ct = chunk_of(t);
      J1 = max(J1, block_end(chunk_visible(a, L, ct), parts_of(ct)));
    }
    if constexpr (wide_mode(MODE)) {
      if (two) {
        const bool has_b = tile + NW < nchunk;
        WA wave_b(a.scale_log2);
        const ChunkRows cb = setup(wave_b, chunk_of(has_b ? tile + NW : tile));
        run_staged<D, kStepBlocks, 2, NW>(wave, wave_b, lds.st, table_row, j_begin, J1, block_end(ca.l_vis, ca.nparts),
                                      has_b ? block_end(cb.l_vis, cb.nparts) : 0, true, 0, 1, L, ca.l_first,
                                      max(ca.l_vis, 0), cb.l_first, max(cb.l_vis, 0), kpool, vpool, block_bytes,
                                      a.num_blocks);
        wave.finish();
        wave_b.finish();
        epilogue(wave, ca.rows, true, 0, NW, 1, any_bad, true);
        __syncthreads();  // the second set reuses the epilogue's LDS
        epilogue(wave_b, cb.rows, has_b, NW, nchunk - NW, 1, any_bad, false);
        return;
      }
    }
    run_staged<D, kStepBlocks, 1, NW>(wave, wave, lds.st, table_row, j_begin, J1, block_end(ca.l_vis, ca.nparts), 0,
                                  slice < slices, slice, slices, L, ca.l_first, max(ca.l_vis, 0), 0, 0, kpool, vpool,
                                  block_bytes, a.num_blocks);
  }
  wave.finish();
  epilogue(wave, ca.rows, true, 0, ntile, slices, any_bad, true);
}

template <int D, int MODE>
__device__ void prefix_item(const StepArgs& a, PassLds<D, MODE>& lds, int pitem) {
  constexpr int NW = waves_of(MODE);
  PassShared<D, NW>& sh = lds.sh;
  using WA = WaveAttention<D>;
  const int Hq = a.num_q_heads;
  const int G = a.group;
  const int g = pitem % a.num_kv_heads;  // pitem = ((group * Pp + pp) * RG + rg) * Hkv + g
  const int RG = a.prefix_row_groups;
  const int rg = (pitem / a.num_kv_heads) % RG;
  const int pp = (pitem / (a.num_kv_heads * RG)) % a.prefix_partitions;
  const int grp = pitem / (a.num_kv_heads * RG * a.prefix_partitions);
  const int tid = threadIdx.x;
  const int lane = tid & (kWaveSize - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);

  // group contents are device data: clamp so that nothing is read or written out of bounds
  const int first_g = min(max(a.group_start[grp], 0), a.num_seqs);
  const int members_g = min(min(a.group_start[grp + 1], a.num_seqs) - first_g, a.max_group_size);
  // this item's row group: members [rg MR, rg MR + MR) of the group (in 64
  // bits: RG MR may pass B by up to MR - 1)
  const int64_t m0 = (int64_t)rg * a.members_per_row_group;
  const int members = (int)min((int64_t)a.members_per_row_group, (int64_t)members_g - m0);
  const int first = members > 0 ? first_g + (int)m0 : first_g;
  int plen = a.group_prefix_len[grp];
  plen = plen < 0 ? 0 : (plen > a.max_prefix_len ? a.max_prefix_len : plen) / kBlockTokens * kBlockTokens;
  const int Tp = a.partition_tokens;
  if (members <= 0 || pp * Tp >= plen) return;
  const int nq = a.num_query_tokens;
  const int rows = members * nq * G;               // member-major, then the new tokens, then the G heads
  const int ntile = (rows + kRows - 1) / kRows;    // 16-row tiles: 1 .. 4
  const int slices = NW / ntile;                   // slices of blocks per tile
  const int tile = w % ntile;
  const int slice = w / ntile;
  const int t_end = min(plen, (pp + 1) * Tp);
  const int j_begin = (pp * Tp) / kBlockTokens;
  const int j_end = t_end / kBlockTokens;
  const int tile_rows = min(kRows, rows - tile * kRows);

  // The prefix tokens row (member m, new token i) sees: those below its own
  // position's limit L_m - n + 1 + i, at most the whole prefix (all of it
  // when the new tokens come after the prefix).
  auto seen = [&](int m, int i) {
    int Lm = a.lens[first + m];
    Lm = Lm < 0 ? 0 : (Lm > a.max_context_len ? a.max_context_len : Lm);
    return min(plen, max(Lm - nq + 1 + i, 0));
  };
  int l_first = plen;  // every row of the item sees the prefix tokens below it
  for (int m = 0; m < members; ++m) l_first = min(l_first, seen(m, 0));
  // lane row n of this tile repeats real rows past the tile's last one
  const int r = tile * kRows + (lane & 15) % tile_rows;
  const int m_r = r / (nq * G), i_r = (r / G) % nq;
  const int b = first + m_r;
  WA wave(a.scale_log2);
  wave.start(a.q + (((size_t)b * nq + i_r) * Hq + (size_t)g * G + r % G) * D, plen - seen(m_r, i_r));
  const char* kpool = reinterpret_cast<const char*>(a.k) + (size_t)g * WA::kTileBytes;
  const char* vpool = reinterpret_cast<const char*>(a.v) + (size_t)g * WA::kTileBytes;
  // the prefix blocks are those of the group's first member (shared by contract)
  const int32_t* table_row = a.table + (size_t)first_g * a.max_blocks_per_seq;
  const size_t block_bytes = (size_t)a.num_kv_heads * WA::kTileBytes;
  if (MODE == kModeRegister && ntile != 1) return;  // not this launch's kind (never: the host picks the mode)
  if (ntile == 1) {  // one tile: the 4 wavefronts split the blocks, tiles into registers
    const int per_slice = (j_end - j_begin + NW - 1) / NW;
    const int wj0 = min(j_end, j_begin + w * per_slice);
    const int wj1 = min(j_end, wj0 + per_slice);
    wave.run(table_row, wj0, wj1, plen, l_first, plen, kpool, vpool, block_bytes, a.num_blocks);
  } else if constexpr (MODE != kModeRegister) {  // several tiles: every block staged once through LDS for all of them
    run_staged<D, kStepBlocks, 1, NW>(wave, wave, lds.st, table_row, j_begin, j_end, j_end, 0, slice < slices, slice,
                                  slices, plen, l_first, plen, 0, 0, kpool, vpool, block_bytes, a.num_blocks);
  }
  wave.finish();
  publish(sh, wave, w, lane, tile_rows);
  __syncthreads();
  row_weights(sh, ntile, slices);

  // ---- merge the slices of each tile in a fixed order; every member row gets a partial state ----
  int any_bad = 0;
#pragma unroll
  for (int x = 0; x < NW; ++x) any_bad |= sh.bad[x];
  for (int idx = tid; idx < rows * (D / 4); idx += NW * kWaveSize) {  // 4 columns per thread
    const int rr = idx / (D / 4);
    const int d0 = 4 * (idx % (D / 4));
    const int t = rr / kRows, h = rr % kRows;
    float acc[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = any_bad ? __builtin_nanf("") : combine(sh, t, ntile, slices, h, d0 + e);
    const size_t row = ((size_t)(first + rr / (nq * G)) * nq + (rr / G) % nq) * Hq + (size_t)g * G + rr % G;
    store_partial4(a, row * a.slots_per_row + pp, d0, D, acc, sh.mx[t][h], sh.lsum[t][h]);
  }
}

// Occupancy: 3 wavefronts per SIMD (12 per compute unit) at most 168 VGPRs;
// the wide variant 2 (256 VGPRs).
template <int D, int MODE>
__global__ void __launch_bounds__(waves_of(MODE) * kWaveSize)
__attribute__((amdgpu_waves_per_eu(wide_mode(MODE) ? 2 : 3)))
partition_kernel(const StepArgs a) {
  __shared__ __align__(16) PassLds<D, MODE> lds;
  const int item = a.order ? a.order[blockIdx.x] : (int)blockIdx.x;  // no order: every item runs at once
  // an order reused from an earlier call is the caller's contract; never step outside the items
  if ((unsigned)item >= (unsigned)(a.num_regular_items + a.num_prefix_items)) return;
  if (item < a.num_regular_items)
    regular_item<D, MODE>(a, lds, item);
  else
    prefix_item<D, MODE>(a, lds, item - a.num_regular_items);
}

template <int D>
hipError_t launch_d(const StepArgs& a, hipStream_t stream) {
  const unsigned grid = (unsigned)a.num_regular_items + (unsigned)a.num_prefix_items;
  // which kinds of items the step has: a regular item has one tile when its
  // chunk group holds one query chunk; a prefix item may have one tile
  // whenever groups exist (a row group can be small) and several when the
  // bound on a row group's rows exceeds one tile
  const bool groups = a.num_groups > 0;
  const bool one = a.num_query_chunks % kWaves == 1 || groups;
  const bool several =
      a.num_query_chunks >= 2 ||
      (groups && (int64_t)min(a.max_group_size, a.members_per_row_group) * a.num_query_tokens * a.group > kRows);
  const dim3 block(kWaves * kWaveSize);
  if (a.chunks_per_group > kWideChunks)
    hipLaunchKernelGGL((partition_kernel<D, kModeWide16>), dim3(grid), dim3(waves_of(kModeWide16) * kWaveSize), 0,
                       stream, a);
  else if (a.chunks_per_group > kWaves)
    hipLaunchKernelGGL((partition_kernel<D, kModeWide>), dim3(grid), block, 0, stream, a);
  else if (one && !several)
    hipLaunchKernelGGL((partition_kernel<D, kModeRegister>), dim3(grid), block, 0, stream, a);
  else
    hipLaunchKernelGGL((partition_kernel<D, kModeMixed>), dim3(grid), block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_partition(const StepArgs& a, int head_dim, hipStream_t stream) {
  if (head_dim == 64) return launch_d<64>(a, stream);
  if (head_dim == 128) return launch_d<128>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace pda
