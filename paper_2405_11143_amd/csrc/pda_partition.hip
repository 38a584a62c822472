// Pass 1: one workgroup per (partition of a context, sequence, KV head,
// chunk of new query tokens), taken in the order pda_order.hip computed
// (largest partition first).
//
// A chunk holds up to 16 / G consecutive new tokens of the sequence, so its
// query rows (token-major, then the G heads of the KV head) fill at most one
// 16-row MFMA tile; a decode step has one token, i.e. one chunk of G rows.
// New token i of a sequence with n new tokens and context length L sits at
// position L - n + i and sees tokens t < L - n + 1 + i.
//
// The partition's 16-token blocks that the chunk can see are split into 4
// contiguous runs, one per wavefront; each wavefront streams its run with
// WaveAttention (pda_wave.h) and the 4 states are merged through LDS in a
// fixed order.  The workgroup leaves the final output rows (the chunk sees a
// single partition) or a partial softmax state (max, denominator,
// unnormalised output) for the merge pass.  Nothing depends on physical
// block ids or on timing, so results are bit-for-bit reproducible and
// independent of block placement.
#include "pda_wave.h"

namespace pda {
namespace {

// Occupancy: 3 wavefronts per SIMD (12 per compute unit) at most 168 VGPRs.
template <int D>
__global__ void __launch_bounds__(kWaves * kWaveSize) __attribute__((amdgpu_waves_per_eu(3)))
partition_kernel(const StepArgs a) {
  using WA = WaveAttention<D>;
  constexpr int kRows = 16;
  __shared__ __align__(16) float s_o[kWaves][kRows][D];
  __shared__ float s_m[kWaves][kRows];
  __shared__ float s_l[kWaves][kRows];
  __shared__ int s_bad[kWaves];

  const int Hq = a.num_q_heads;
  const int G = a.group;
  const int HC = a.num_kv_heads * a.num_query_chunks;
  const int item = a.order[blockIdx.x];  // (p * B + b) * HC + g * NQC + chunk
  const int gc = item % HC;
  const int b = (item / HC) % a.num_seqs;
  const int p = item / (HC * a.num_seqs);
  const int g = gc / a.num_query_chunks;
  const int chunk = gc % a.num_query_chunks;
  const int nq = a.num_query_tokens;
  const int i0 = chunk * a.query_chunk;                // first new token of the chunk
  const int nv = min(a.query_chunk, nq - i0);          // its tokens
  const int rows = nv * G;                             // its query rows, token-major
  const int tid = threadIdx.x;
  const int lane = tid & (kWaveSize - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  auto out_row = [&](int r) {  // output row of chunk row r
    return ((size_t)b * nq + i0 + r / G) * Hq + (size_t)g * G + r % G;
  };

  int L = a.lens[b];
  L = L < 0 ? 0 : (L > a.max_context_len ? a.max_context_len : L);
  const int l_vis = chunk_visible(a, L, chunk);  // the chunk's last row sees tokens below this
  const int l_first = l_vis - nv + 1;  // its first row sees tokens below this
  if (l_vis <= 0) {
    if (p == 0)
      for (int i = tid; i < rows * D; i += kWaves * kWaveSize) a.out[out_row(i / D) * D + i % D] = 0.f;
    return;
  }
  const int Tp = a.partition_tokens;
  const int nparts = (l_vis + Tp - 1) / Tp;
  if (p >= nparts) return;
  const int t_end = min(l_vis, (p + 1) * Tp);
  const int j_begin = (p * Tp) / kBlockTokens;
  const int j_end = (t_end + kBlockTokens - 1) / kBlockTokens;
  const int per_wave = (j_end - j_begin + kWaves - 1) / kWaves;
  const int wj0 = min(j_end, j_begin + w * per_wave);
  const int wj1 = min(j_end, wj0 + per_wave);

  // lane row n repeats real rows past the chunk's last one
  const int r = (lane & 15) % rows;
  const int qi = i0 + r / G;
  WA wave(a.scale_log2);
  wave.start(a.q + (((size_t)b * nq + qi) * Hq + (size_t)g * G + r % G) * D, nq - 1 - qi);
  const char* kpool = reinterpret_cast<const char*>(a.k) + (size_t)g * WA::kTileBytes;
  const char* vpool = reinterpret_cast<const char*>(a.v) + (size_t)g * WA::kTileBytes;
  wave.run(a.table + (size_t)b * a.max_blocks_per_seq, wj0, wj1, L, l_first, l_vis, kpool, vpool,
           (size_t)a.num_kv_heads * WA::kTileBytes, a.num_blocks);
  wave.finish();

  const int n = lane & 15;
  if (n < rows) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (D == 128) {
        const int d0 = wave.d_of(i, 0);  // 8 consecutive columns
        *reinterpret_cast<float4*>(&s_o[w][n][d0]) =
            make_float4(wave.o[0][i], wave.o[1][i], wave.o[2][i], wave.o[3][i]);
        *reinterpret_cast<float4*>(&s_o[w][n][d0 + 4]) =
            make_float4(wave.o[4][i], wave.o[5][i], wave.o[6][i], wave.o[7][i]);
      } else {
        const int d0 = wave.d_of(i, 0);  // 4 consecutive columns
        *reinterpret_cast<float4*>(&s_o[w][n][d0]) =
            make_float4(wave.o[0][i], wave.o[1][i], wave.o[2][i], wave.o[3][i]);
      }
    }
    if (lane < 16) {
      s_m[w][n] = wave.m_run;
      s_l[w][n] = wave.l_run;
    }
  }
  if (lane == 0) s_bad[w] = wave.bad ? 1 : 0;
  __syncthreads();

  // ---- merge the 4 wavefront states in a fixed order ----
  int any_bad = 0;
#pragma unroll
  for (int x = 0; x < kWaves; ++x) any_bad |= s_bad[x];
  const bool single = nparts == 1;
  for (int idx = tid; idx < rows * D; idx += kWaves * kWaveSize) {
    const int h = idx / D;
    const int d = idx % D;
    float M = WA::kFloor;
#pragma unroll
    for (int x = 0; x < kWaves; ++x) M = fmaxf(M, s_m[x][h]);
    float acc = 0.f, lsum = 0.f;
#pragma unroll
    for (int x = 0; x < kWaves; ++x) {
      const float sc = exp2_fast(s_m[x][h] - M);  // 0 for a wavefront without tokens of this row
      acc = fmaf(sc, s_o[x][h][d], acc);
      lsum = fmaf(sc, s_l[x][h], lsum);
    }
    if (any_bad) acc = __builtin_nanf("");
    const size_t row = out_row(h);
    if (single) {
      a.out[row * D + d] = lsum > 0.f ? acc / lsum : acc;  // acc is 0 (or NaN) for a row that sees nothing
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

template <int D>
hipError_t launch_d(const StepArgs& a, hipStream_t stream) {
  const unsigned grid = (unsigned)a.num_partitions * (unsigned)a.num_seqs * (unsigned)a.num_kv_heads *
                        (unsigned)a.num_query_chunks;
  hipLaunchKernelGGL((partition_kernel<D>), dim3(grid), dim3(kWaves * kWaveSize), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_partition(const StepArgs& a, int head_dim, hipStream_t stream) {
  if (head_dim == 64) return launch_d<64>(a, stream);
  if (head_dim == 128) return launch_d<128>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace pda
