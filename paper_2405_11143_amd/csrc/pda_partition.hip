// Pass 1 of paged decode attention on gfx950: one workgroup per
// (partition of a context, sequence, KV head).
//
// What is computed: single-query attention over a paged KV cache with
// grouped-query heads -- the rollout decode step the paper runs through
// vLLM's PagedAttention (Section 3.2; Appendix C, rollout generation).  Each
// workgroup handles the G query heads that share one KV head over a range of
// `partition_tokens` logical tokens of one sequence, and leaves either the
// final output rows (context fits one partition) or a partial softmax state
// (max, denominator, unnormalised output) for the merge pass.
//
// Mapping onto CDNA4 (64-wide wavefronts, MFMA, LDS):
//  * The partition's 16-token blocks are split into 4 contiguous runs, one per
//    wavefront; each wavefront keeps its own online-softmax state and
//    prefetches the next block's K and V tiles (2 x 16 x D bf16) into
//    registers while it computes on the current one.  Every tile load is a
//    buffer load (descriptor = the tile, so no read can leave it) whose
//    instruction reads 1 KiB of contiguous memory (whole cache lines) with
//    the non-temporal hint: the cache is streamed once, and measured on MI355X
//    the hint lifts a plain 4 KiB-tile gather from ~6.1 to ~6.9 TB/s.  All K
//    and V loads of a lane share one 32-bit offset register.
//  * Scores S[G][16] = Q_g K^T are one small dense contraction per block:
//    D/32 MFMA f32_16x16x32_bf16 with the G query heads (repeated to fill 16
//    rows) as the A operand and the K tile as the B operand.  The K cache
//    stores each block as D/8 chunks of [16 slots][8 elements], so the B
//    fragment of lane l in k-step c -- 8 consecutive d of token l%16, chunk
//    4c + l/16 -- is exactly the 16 bytes at offset 1024c + 16l of the tile:
//    K goes from HBM straight into MFMA registers with fully contiguous
//    loads.  The A operand (q) uses the same assignment of d to (k-step,
//    k-group, element), so the contraction is unchanged.
//  * The online softmax runs on the MFMA output layout: a lane holds the
//    scores of 4 head rows for one token.  The running maximum is moved only
//    when some score of the block exceeds it by more than 2^8 (a wavefront
//    vote); then the block max of each row is a 16-lane all-reduce of four
//    DPP moves (quad swaps, half-row and row mirror) and the state is
//    rescaled.  Otherwise probabilities are taken against the stale maximum
//    (they stay below 2^8, far inside fp32), so most blocks need neither the
//    reduction nor the O rescale; the result is the same softmax.  Each lane
//    accumulates the denominator of its own token column; columns are summed
//    once, at the end.
//  * P V runs on the VALU in fp32: lane (phase, chunk) owns 8 consecutive d
//    for all G heads and the tokens of its phase, so each V load instruction
//    reads 1 KiB of contiguous tile.  The probabilities and rescale factors
//    of a block travel from the MFMA layout to this layout through LDS
//    (double-buffered per wavefront; only a wavefront barrier is needed).
//  * Tokens past the context in the last block are removed by selection, not
//    by multiplying with zero, so whatever those slots hold (NaN included)
//    never reaches the result.
//  * The 4 wavefront states are merged through LDS in a fixed order.  Nothing
//    depends on physical block ids or on timing, so results are bit-for-bit
//    reproducible and independent of block placement.
#include "pda_internal.h"

namespace pda {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));

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

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

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

// Occupancy: up to G = 8 the kernel fits 168 VGPRs, i.e. 3 wavefronts per
// SIMD (12 per compute unit); the hint makes the compiler hold that line for
// G = 8, which would otherwise take 170 registers and drop to 2.
template <int G, int D>
__global__ void __launch_bounds__(kWaves * kWaveSize) __attribute__((amdgpu_waves_per_eu(G <= 8 ? 3 : 1)))
partition_kernel(const StepArgs a) {
  static_assert(G >= 1 && G <= kMaxGroup, "query heads per KV head");
  static_assert(D == 64 || D == 128, "head_dim");
  constexpr int NC = D / 32;                 // MFMA k-steps per block
  constexpr int CPR = D / 8;                 // 16-byte chunks per K/V row
  constexpr int NPH = kWaveSize / CPR;       // token phases of the P.V layout
  constexpr int TPL = kBlockTokens / NPH;    // tokens per lane per block in P.V
  constexpr int GP = (G + 3) & ~3;           // head count padded to float4
  constexpr float kNegInf = -__builtin_huge_valf();
  constexpr float kRescaleSlack = 8.f;       // log2 of the largest unnormalised probability

  __shared__ __align__(16) float s_p[kWaves][2][kBlockTokens][GP];
  __shared__ __align__(16) float s_alpha[kWaves][2][GP];
  __shared__ __align__(16) float s_o[kWaves][G][D];
  __shared__ float s_m[kWaves][GP];
  __shared__ float s_l[kWaves][GP];
  __shared__ int s_bad[kWaves];

  const int Hkv = a.num_kv_heads;
  const int Hq = a.num_q_heads;
  const int item = blockIdx.x;
  const int g = item % Hkv;
  const int b = (item / Hkv) % a.num_seqs;
  const int p = item / (Hkv * a.num_seqs);
  const int tid = threadIdx.x;
  const int lane = tid & (kWaveSize - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int head0 = g * G;

  int L = a.lens[b];
  L = L < 0 ? 0 : (L > a.max_context_len ? a.max_context_len : L);
  if (L == 0) {
    if (p == 0) {
      float* o = a.out + ((size_t)b * Hq + head0) * D;
      for (int i = tid; i < G * D; i += kWaves * kWaveSize) o[i] = 0.f;
    }
    return;
  }
  const int Tp = a.partition_tokens;
  const int nparts = (L + Tp - 1) / Tp;
  if (p >= nparts) return;
  const int t_end = min(L, (p + 1) * Tp);
  const int j_begin = (p * Tp) / kBlockTokens;
  const int j_end = (t_end + kBlockTokens - 1) / kBlockTokens;
  const int per_wave = (j_end - j_begin + kWaves - 1) / kWaves;
  const int wj0 = min(j_end, j_begin + w * per_wave);
  const int wj1 = min(j_end, wj0 + per_wave);

  // MFMA fragment coordinates: n = row of A (head) / column of B (token),
  // kg = k-group; in k-step c the lane's 8 reduction indices are
  // d = 8 * (4c + kg) + e, e < 8 (chunk 4c + kg of the K tile).
  const int n = lane & 15;
  const int kg = lane >> 4;
  // P.V coordinates: this lane owns d in [8*(lane % CPR), +8) for the tokens
  // tp, tp + NPH, ... of each block.
  const int tp = lane / CPR;

  // A operand: query head (n mod G) of this KV head, d = 32c + 8kg + e.
  bf16x8_t qa[NC];
  {
    const uint16_t* qrow = a.q + ((size_t)b * Hq + head0 + (n % G)) * D + kg * 8;
#pragma unroll
    for (int c = 0; c < NC; ++c)
      qa[c] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(qrow + 32 * c));
  }

  constexpr int kTileBytes = kBlockTokens * D * 2;                // one (block, KV head) tile
  const size_t block_bytes = (size_t)Hkv * kTileBytes;              // one pool block, all heads
  const char* kpool = reinterpret_cast<const char*>(a.k) + (size_t)g * kTileBytes;
  const char* vpool = reinterpret_cast<const char*>(a.v) + (size_t)g * kTileBytes;
  // K: lane l's fragment for k-step c is the 16 bytes at 1024c + 16l of the
  // tile.  V: the same offsets hold row NPH*i + tp, columns 8*(lane % CPR) + e.
  const int lane_off = lane * 16;
  const int32_t* trow = a.table + (size_t)b * a.max_blocks_per_seq;
  bool bad = false;

  // Block ids of this wavefront's run, one per lane (64 blocks at a time), so
  // the loop never waits on a scalar load before issuing a tile load.
  int ids = 0;
  auto fetch_ids = [&](int first) {
    const int j = first + lane;
    ids = j < wj1 ? trow[j] : 0;
  };
  auto load_tiles = [&](uint4 (&kr)[NC], uint4 (&vr)[TPL], int i, bool needed) {
    int phys = __builtin_amdgcn_readlane(ids, i);
    if ((unsigned)phys >= (unsigned)a.num_blocks) {  // contract violation: never read outside the pool
      bad = true;
      phys = 0;
    }
    const size_t off = (size_t)phys * block_bytes;
    const int bytes = needed ? kTileBytes : 0;
    const __amdgpu_buffer_rsrc_t rk = tile_rsrc(kpool + off, bytes);
    const __amdgpu_buffer_rsrc_t rv = tile_rsrc(vpool + off, bytes);
#pragma unroll
    for (int c = 0; c < NC; ++c) kr[c] = load_stream(rk, lane_off + c * 1024);
#pragma unroll
    for (int i2 = 0; i2 < TPL; ++i2) vr[i2] = load_stream(rv, lane_off + i2 * 1024);
  };

  float o[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[h][e] = 0.f;
  float m_run[4], l_run[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    m_run[i] = kNegInf;
    l_run[i] = 0.f;
  }

  auto process = [&](const uint4 (&kr)[NC], const uint4 (&vr)[TPL], int j, int par) {
    // ---- scores: S = Q_g K^T on MFMA; lane holds rows 4*kg+i, column n ----
    floatx4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NC; ++c)
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[c], __builtin_bit_cast(bf16x8_t, kr[c]), acc, 0, 0, 0);
    const bool tail = (j + 1) * kBlockTokens > L;  // wave-uniform
    const int tok0 = j * kBlockTokens;
    float sc[4];
    bool grow = false;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sc[i] = acc[i] * a.scale_log2;
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
      *reinterpret_cast<float4*>(&s_p[w][par][n][4 * kg]) = make_float4(pr[0], pr[1], pr[2], pr[3]);
      if (rescale && n == 0)
        *reinterpret_cast<float4*>(&s_alpha[w][par][4 * kg]) = make_float4(al[0], al[1], al[2], al[3]);
    }
    wave_lds_sync();

    // ---- O = alpha * O + P V on the VALU ----
    if (rescale) {
      float alpha[GP];
#pragma unroll
      for (int h4 = 0; h4 < GP; h4 += 4) {
        const float4 t = *reinterpret_cast<const float4*>(&s_alpha[w][par][h4]);
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
        const float4 t = *reinterpret_cast<const float4*>(&s_p[w][par][row][h4]);
        ph[h4] = t.x; ph[h4 + 1] = t.y; ph[h4 + 2] = t.z; ph[h4 + 3] = t.w;
      }
#pragma unroll
      for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) o[h][e] = fmaf(ph[h], f[e], o[h][e]);
    }
  };

  {
    // Two register buffers: the tiles of block i+1 are in flight while block i
    // is computed.  Every load is unconditional, so the compiler counts
    // outstanding loads exactly and waits only for the tiles it is about to
    // use; the scheduling barriers keep each prefetch ahead of the first use
    // of the current tiles.  Past the end of the run the prefetch gets a
    // zero-length descriptor: the hardware drops it without touching memory.
    // Block ids come in chunks of 64, one per lane.
    const int cnt = wj1 - wj0;
    uint4 k0[NC], v0[TPL], k1[NC], v1[TPL];
    for (int c0 = 0; c0 < cnt; c0 += kWaveSize) {
      const int cn = min(kWaveSize, cnt - c0);
      const int jc = wj0 + c0;
      fetch_ids(jc);
      load_tiles(k0, v0, 0, true);
      for (int i = 0; i < cn; i += 2) {
        load_tiles(k1, v1, min(i + 1, cn - 1), i + 1 < cn);
        __builtin_amdgcn_sched_barrier(0);
        process(k0, v0, jc + i, 0);
        if (i + 1 >= cn) break;
        load_tiles(k0, v0, min(i + 2, cn - 1), i + 2 < cn);
        __builtin_amdgcn_sched_barrier(0);
        process(k1, v1, jc + i + 1, 1);
      }
    }
  }

  // ---- wavefront state: sum denominators over token columns, O over phases ----
#pragma unroll
  for (int i = 0; i < 4; ++i) l_run[i] = row16_sum(l_run[i]);
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e)
#pragma unroll
      for (int x = CPR; x < kWaveSize; x <<= 1) o[h][e] += __shfl_xor(o[h][e], x);

  if (lane < CPR) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      *reinterpret_cast<float4*>(&s_o[w][h][8 * lane]) = make_float4(o[h][0], o[h][1], o[h][2], o[h][3]);
      *reinterpret_cast<float4*>(&s_o[w][h][8 * lane + 4]) = make_float4(o[h][4], o[h][5], o[h][6], o[h][7]);
    }
  }
  if (n == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 4 * kg + i;
      if (r < G) {
        s_m[w][r] = m_run[i];
        s_l[w][r] = l_run[i];
      }
    }
  }
  if (lane == 0) s_bad[w] = bad ? 1 : 0;
  __syncthreads();

  // ---- merge the 4 wavefront states in a fixed order ----
  const bool any_bad = (s_bad[0] | s_bad[1] | s_bad[2] | s_bad[3]) != 0;
  const bool single = nparts == 1;
  for (int idx = tid; idx < G * D; idx += kWaves * kWaveSize) {
    const int h = idx / D;
    const int d = idx % D;
    float M = kNegInf;
#pragma unroll
    for (int x = 0; x < kWaves; ++x) M = fmaxf(M, s_m[x][h]);
    float acc = 0.f, lsum = 0.f;
#pragma unroll
    for (int x = 0; x < kWaves; ++x) {
      const float sc = exp2_fast(s_m[x][h] - M);  // 0 for a wavefront without tokens
      acc = fmaf(sc, s_o[x][h][d], acc);
      lsum = fmaf(sc, s_l[x][h], lsum);
    }
    if (any_bad) acc = __builtin_nanf("");
    const size_t row = (size_t)b * Hq + head0 + h;
    if (single) {
      a.out[row * D + d] = acc / lsum;
    } else {
      const size_t slot = row * a.num_partitions + p;
      a.part_o[slot * D + d] = acc;
      if (d == 0) {
        a.part_m[slot] = M;
        a.part_l[slot] = lsum;
      }
    }
  }
}

template <int G, int D>
hipError_t launch_gd(const StepArgs& a, hipStream_t stream) {
  const unsigned grid = (unsigned)a.num_partitions * (unsigned)a.num_seqs * (unsigned)a.num_kv_heads;
  hipLaunchKernelGGL((partition_kernel<G, D>), dim3(grid), dim3(kWaves * kWaveSize), 0, stream, a);
  return hipGetLastError();
}

template <int D>
hipError_t launch_d(const StepArgs& a, int group, hipStream_t stream) {
  switch (group) {
    case 1: return launch_gd<1, D>(a, stream);
    case 2: return launch_gd<2, D>(a, stream);
    case 3: return launch_gd<3, D>(a, stream);
    case 4: return launch_gd<4, D>(a, stream);
    case 5: return launch_gd<5, D>(a, stream);
    case 6: return launch_gd<6, D>(a, stream);
    case 7: return launch_gd<7, D>(a, stream);
    case 8: return launch_gd<8, D>(a, stream);
    case 9: return launch_gd<9, D>(a, stream);
    case 10: return launch_gd<10, D>(a, stream);
    case 11: return launch_gd<11, D>(a, stream);
    case 12: return launch_gd<12, D>(a, stream);
    case 13: return launch_gd<13, D>(a, stream);
    case 14: return launch_gd<14, D>(a, stream);
    case 15: return launch_gd<15, D>(a, stream);
    case 16: return launch_gd<16, D>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_partition(const StepArgs& a, int group, int head_dim, hipStream_t stream) {
  if (head_dim == 64) return launch_d<64>(a, group, stream);
  if (head_dim == 128) return launch_d<128>(a, group, stream);
  return hipErrorInvalidValue;
}

}  // namespace pda
