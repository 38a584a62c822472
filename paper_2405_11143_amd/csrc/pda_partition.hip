// Pass 1: one workgroup per (partition of a context, sequence, KV head),
// taken in the order pda_order.hip computed (largest partition first).
//
// The partition's 16-token blocks are split into 4 contiguous runs, one per
// wavefront; each
// wavefront streams its run with WaveAttention (pda_wave.h) and the 4 states
// are merged through LDS in a fixed order.  The workgroup leaves the final
// output rows (context fits one partition) or a partial softmax state (max,
// denominator, unnormalised output) for the merge pass.  Nothing depends on
// physical block ids or on timing, so results are bit-for-bit reproducible
// and independent of block placement.
#include "pda_wave.h"

namespace pda {
namespace {

// Occupancy: up to G = 8 the kernel fits 168 VGPRs, i.e. 3 wavefronts per
// SIMD (12 per compute unit); the hint makes the compiler hold that line for
// G = 8, which would otherwise take 170 registers and drop to 2.
template <int G, int D>
__global__ void __launch_bounds__(kWaves * kWaveSize) __attribute__((amdgpu_waves_per_eu(G <= 8 ? 3 : 1)))
partition_kernel(const StepArgs a) {
  using WA = WaveAttention<G, D>;
  __shared__ __align__(16) typename WA::Exchange s_x[kWaves];
  __shared__ __align__(16) float s_o[kWaves][G][D];
  __shared__ float s_m[kWaves][G];
  __shared__ float s_l[kWaves][G];
  __shared__ int s_bad[kWaves];

  const int Hkv = a.num_kv_heads;
  const int Hq = a.num_q_heads;
  const int item = a.order[blockIdx.x];  // (p * B + b) * Hkv + g
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

  WA wave(&s_x[w], a.scale_log2);
  wave.start(a.q + ((size_t)b * Hq + head0) * D);
  const char* kpool = reinterpret_cast<const char*>(a.k) + (size_t)g * WA::kTileBytes;
  const char* vpool = reinterpret_cast<const char*>(a.v) + (size_t)g * WA::kTileBytes;
  wave.run(a.table + (size_t)b * a.max_blocks_per_seq, wj0, wj1, L, kpool, vpool,
           (size_t)Hkv * WA::kTileBytes, a.num_blocks);
  wave.finish();

  if (lane < WA::CPR) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      *reinterpret_cast<float4*>(&s_o[w][h][8 * lane]) =
          make_float4(wave.o[h][0], wave.o[h][1], wave.o[h][2], wave.o[h][3]);
      *reinterpret_cast<float4*>(&s_o[w][h][8 * lane + 4]) =
          make_float4(wave.o[h][4], wave.o[h][5], wave.o[h][6], wave.o[h][7]);
    }
  }
  if (lane == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      s_m[w][h] = wave.mh[h];
      s_l[w][h] = wave.lh[h];
    }
    s_bad[w] = wave.bad ? 1 : 0;
  }
  __syncthreads();

  // ---- merge the 4 wavefront states in a fixed order ----
  int any_bad = 0;
#pragma unroll
  for (int x = 0; x < kWaves; ++x) any_bad |= s_bad[x];
  const bool single = nparts == 1;
  for (int idx = tid; idx < G * D; idx += kWaves * kWaveSize) {
    const int h = idx / D;
    const int d = idx % D;
    float M = WA::kNegInf;
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

}  // namespace

hipError_t launch_partition(const StepArgs& a, int group, int head_dim, hipStream_t stream) {
  return dispatch_gd(group, head_dim, [&](auto gt, auto dt) {
    return launch_gd<decltype(gt)::value, decltype(dt)::value>(a, stream);
  });
}

}  // namespace pda
