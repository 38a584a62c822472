// Pass 1, stream schedule (the default): the whole step's work is cut into
// equal contiguous shares, one per resident wavefront.
//
// Work is the sequence of (sequence b, KV head g, 16-token block j) in that
// order; it has T = Hkv * sum_b ceil(L_b / 16) blocks.  Wavefront v of
// V = min(workers, T) takes blocks [floor(vT/V), floor((v+1)T/V)) -- never
// empty -- whatever sequence boundaries fall inside, and streams each (b, g) piece of its share -- a segment --
// with WaveAttention (pda_wave.h).  V is the number of wavefronts the GPU
// holds at once, so every wavefront starts at launch, streams for the whole
// kernel without a workgroup barrier, and all finish together: there is no
// tail of partial workgroups and no per-item start-up, which on MI355X is
// what separates a per-partition grid from the HBM read ceiling on ragged
// batches.
//
// A segment that covers a whole (b, g) writes the final output rows; the
// others write a partial softmax state at slot (b*Hkv + g) + v (unique:
// along the work order the unit index and the wavefront index never both
// stay the same from one segment to the next), and the first segment of each
// (b, g) records (its wavefront, number of segments) for the merge pass.
// Segment boundaries depend only on the lengths and on V, never on physical
// block ids or timing, so results are bit-for-bit reproducible and
// independent of block placement.
#include "pda_wave.h"

namespace pda {
namespace {

template <int G, int D>
__global__ void __launch_bounds__(kWaves * kWaveSize) __attribute__((amdgpu_waves_per_eu(G <= 8 ? 3 : 1)))
stream_kernel(const StepArgs a) {
  using WA = WaveAttention<G, D>;
  extern __shared__ int s_pre[];  // [B + 1]: blocks of sequences before b
  __shared__ __align__(16) typename WA::Exchange s_x[kWaves];
  __shared__ int s_wsum[kWaves];

  const int B = a.num_seqs;
  const int Hkv = a.num_kv_heads;
  const int Hq = a.num_q_heads;
  const int tid = threadIdx.x;
  const int lane = tid & (kWaveSize - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  auto clamp_len = [&](int L) { return L < 0 ? 0 : (L > a.max_context_len ? a.max_context_len : L); };

  // ---- prefix sums of per-sequence block counts (every workgroup) ----
  for (int i = tid; i < B; i += kWaves * kWaveSize) s_pre[i] = (clamp_len(a.lens[i]) + kBlockTokens - 1) / kBlockTokens;
  __syncthreads();
  const int per = (B + kWaves * kWaveSize - 1) / (kWaves * kWaveSize);
  const int b0 = min(B, tid * per), b1 = min(B, b0 + per);
  int local = 0;
  for (int i = b0; i < b1; ++i) local += s_pre[i];
  int inc = local;
  for (int o = 1; o < kWaveSize; o <<= 1) {
    const int t = __shfl_up(inc, o);
    if (lane >= o) inc += t;
  }
  if (lane == kWaveSize - 1) s_wsum[w] = inc;
  __syncthreads();
  int run = inc - local;
  for (int x = 0; x < w; ++x) run += s_wsum[x];
  for (int i = b0; i < b1; ++i) {
    const int c = s_pre[i];
    s_pre[i] = run;
    run += c;
  }
  if (tid == 0) {
    int total = 0;
    for (int x = 0; x < kWaves; ++x) total += s_wsum[x];
    s_pre[B] = total;
  }
  __syncthreads();

  // Sequences without tokens get zero rows (no wavefront visits them).
  if (blockIdx.x == 0) {
    for (int bb = 0; bb < B; ++bb)
      if (s_pre[bb + 1] == s_pre[bb]) {
        float* o = a.out + (size_t)bb * Hq * D;
        for (int i = tid; i < Hq * D; i += kWaves * kWaveSize) o[i] = 0.f;
      }
  }

  // ---- this wavefront's share of the work ----
  // With V <= T shares every share is non-empty, so the shares that touch a
  // (b, g) are consecutive wavefronts and the merge can count them.
  const long long T = (long long)Hkv * s_pre[B];
  const long long V = min((long long)a.num_workers, T);
  const int v = blockIdx.x * kWaves + w;
  if (v >= V) return;  // no workgroup barrier follows
  const long long start = (long long)v * T / V;
  const long long end = (long long)(v + 1) * T / V;
  auto wave_of = [&](long long x) { return (int)(((x + 1) * V - 1) / T); };  // share holding block x

  int lo = 0, hi = B - 1;  // last sequence whose blocks start at or before `start`
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if ((long long)Hkv * s_pre[mid] <= start) lo = mid; else hi = mid - 1;
  }
  // Segment state is wave-uniform: keep it in scalar registers.
  auto uni = [](int x) { return __builtin_amdgcn_readfirstlane(x); };
  int b = uni(lo);
  int nb = uni(s_pre[b + 1] - s_pre[b]);
  const long long off = start - (long long)Hkv * s_pre[b];
  int g = uni((int)(off / nb));
  int j = uni((int)(off % nb));
  int rem = uni((int)(end - start));  // a share is < 2^31 blocks

  WA wave(&s_x[w], a.scale_log2);
  const size_t block_bytes = (size_t)Hkv * WA::kTileBytes;
  while (true) {
    const int seg = min(nb - j, rem);
    const int L = uni(clamp_len(a.lens[b]));
    const int u = b * Hkv + g;
    wave.start(a.q + ((size_t)b * Hq + g * G) * D);
    const char* kpool = reinterpret_cast<const char*>(a.k) + (size_t)g * WA::kTileBytes;
    const char* vpool = reinterpret_cast<const char*>(a.v) + (size_t)g * WA::kTileBytes;
    wave.run(a.table + (size_t)b * a.max_blocks_per_seq, j, j + seg, L, kpool, vpool, block_bytes, a.num_blocks);
    wave.finish();
    const float nan = __builtin_nanf("");
    if (j == 0 && seg == nb) {  // the whole (b, g): final rows
      if (lane < WA::CPR) {
        float* orow = a.out + ((size_t)b * Hq + g * G) * D + 8 * lane;
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float r = wave.bad ? nan : 1.f / wave.lh[h];  // exact when l == 1 (one token)
          *reinterpret_cast<float4*>(orow + h * D) =
              make_float4(wave.o[h][0] * r, wave.o[h][1] * r, wave.o[h][2] * r, wave.o[h][3] * r);
          *reinterpret_cast<float4*>(orow + h * D + 4) =
              make_float4(wave.o[h][4] * r, wave.o[h][5] * r, wave.o[h][6] * r, wave.o[h][7] * r);
        }
      }
    } else {  // a piece of (b, g): partial state for the merge pass
      const size_t slot = (size_t)u + v;
      if (lane < WA::CPR) {
        float* po = a.part_o + slot * G * D + 8 * lane;
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float z = wave.bad ? nan : 0.f;
          *reinterpret_cast<float4*>(po + h * D) = make_float4(
              wave.o[h][0] + z, wave.o[h][1] + z, wave.o[h][2] + z, wave.o[h][3] + z);
          *reinterpret_cast<float4*>(po + h * D + 4) = make_float4(
              wave.o[h][4] + z, wave.o[h][5] + z, wave.o[h][6] + z, wave.o[h][7] + z);
        }
      }
      if (lane == 0) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
          a.part_m[slot * G + h] = wave.mh[h];
          a.part_l[slot * G + h] = wave.lh[h];
        }
      }
    }
    if (j == 0 && lane == 0) {
      const long long unit_start = (long long)Hkv * s_pre[b] + (long long)g * nb;
      a.unit_info[2 * u] = v;
      a.unit_info[2 * u + 1] = wave_of(unit_start + nb - 1) - v + 1;
    }
    rem -= seg;
    if (rem == 0) break;
    j = 0;
    if (++g == Hkv) {
      g = 0;
      do { ++b; } while (s_pre[b + 1] == s_pre[b]);  // rem > 0: a sequence with blocks follows
      b = uni(b);
      nb = uni(s_pre[b + 1] - s_pre[b]);
    }
  }
}

template <int G, int D>
hipError_t launch_gd(const StepArgs& a, hipStream_t stream) {
  const unsigned grid = (unsigned)(a.num_workers / kWaves);
  hipLaunchKernelGGL((stream_kernel<G, D>), dim3(grid), dim3(kWaves * kWaveSize), stream_lds_bytes(a.num_seqs),
                     stream, a);
  return hipGetLastError();
}

}  // namespace

size_t stream_lds_bytes(int num_seqs) { return (size_t)(num_seqs + 1) * sizeof(int); }

hipError_t stream_blocks_per_cu(int group, int head_dim, int num_seqs, int* blocks) {
  return dispatch_gd(group, head_dim, [&](auto gt, auto dt) {
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(
        blocks, reinterpret_cast<const void*>(&stream_kernel<decltype(gt)::value, decltype(dt)::value>),
        kWaves * kWaveSize, stream_lds_bytes(num_seqs));
  });
}

hipError_t launch_stream(const StepArgs& a, int group, int head_dim, hipStream_t stream) {
  return dispatch_gd(group, head_dim, [&](auto gt, auto dt) {
    return launch_gd<decltype(gt)::value, decltype(dt)::value>(a, stream);
  });
}

}  // namespace pda
