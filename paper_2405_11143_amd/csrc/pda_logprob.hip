// Token log-probabilities and entropies of one decode step's LM-head logits:
// the rollout records the log-probability of every sampled token, and the
// policy loss uses the entropy of the same distribution (Appendix C).
//
// With x_j = logits[r][j] / T over the vocabulary:
//   logprob[r] = x_tok - log sum_j e^{x_j},  entropy[r] = -sum_j p_j log p_j.
//
// One 1024-thread workgroup streams one row once; the row (250-300 KB for
// Llama-3 / Qwen vocabularies in bf16) is read with 16-byte non-temporal
// buffer loads (descriptor = the row, so no read leaves it), four in flight
// per thread.  Each thread keeps an online state:
//   m   running max of the raw logits,
//   s = sum 2^{d},  t = sum 2^{d} d,  d = (logit - m) * log2(e) / T <= 0,
// rescaled when m grows.  Differences are taken on the raw logits and only
// then scaled, so a large common offset (logits of +-30000, say) costs no
// precision; t is relative to m, so t / s stays small and the entropy keeps
// its precision in fp32.  The states are combined over the workgroup in a
// fixed order (a wavefront butterfly, then the 16 wavefronts in index
// order), so results are reproducible.  Finally
//   logprob = ln2 ((logit_tok - m) log2(e) / T - log2 s),  entropy = ln2 (log2 s - t / s).
// Elements past the vocabulary have probability 0 by selection; -inf logits
// get 2^{-inf} = 0 and add nothing to t.  A token id outside [0, vocab) gives
// NaN.  The inverse temperature must be >= 0 (the host checks it).
#include "pda_internal.h"

namespace pda {
namespace {

constexpr int kLpThreads = 1024;
constexpr int kLpUnroll = 4;  // 16-byte loads in flight per thread
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kFloorMax = -1e30f;  // running max (raw logit units) before any finite logit

struct LpState {
  float m, s, t;
};

// Merge two states; k = log2(e) / T converts raw logit differences.
__device__ __forceinline__ LpState lp_merge(LpState a, LpState b, float k) {
  const float M = fmaxf(a.m, b.m);
  const float da = (a.m - M) * k, db = (b.m - M) * k;  // <= 0
  const float fa = __builtin_amdgcn_exp2f(da);
  const float fb = __builtin_amdgcn_exp2f(db);
  // sum p (d relative to M) = sum p (d relative to m) + (m - M) k sum p, rescaled to M
  LpState r;
  r.m = M;
  r.s = a.s * fa + b.s * fb;
  r.t = (a.s > 0.f ? (a.t + da * a.s) * fa : 0.f) + (b.s > 0.f ? (b.t + db * b.s) * fb : 0.f);
  return r;
}

template <int ESIZE>
__device__ __forceinline__ void unpack(const uint4 u, float (&f)[16 / ESIZE]) {
  if (ESIZE == 2) {
    f[0] = __uint_as_float(u.x << 16);
    f[1] = __uint_as_float(u.x & 0xffff0000u);
    f[2] = __uint_as_float(u.y << 16);
    f[3] = __uint_as_float(u.y & 0xffff0000u);
    f[4] = __uint_as_float(u.z << 16);
    f[5] = __uint_as_float(u.z & 0xffff0000u);
    f[6] = __uint_as_float(u.w << 16);
    f[7] = __uint_as_float(u.w & 0xffff0000u);
  } else {
    f[0] = __uint_as_float(u.x);
    f[1] = __uint_as_float(u.y);
    f[2] = __uint_as_float(u.z);
    f[3] = __uint_as_float(u.w);
  }
}

// ESIZE: bytes per logit (2 = bf16, 4 = fp32).
template <int ESIZE>
__global__ void __launch_bounds__(kLpThreads) logprob_kernel(const LogprobArgs a) {
  constexpr int E = 16 / ESIZE;  // logits per 16-byte load
  __shared__ LpState s_state[kLpThreads / kWaveSize];
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  const char* base = static_cast<const char*>(a.logits) + (size_t)row * a.row_stride * ESIZE;
  // The descriptor covers the vocabulary rounded up to 16 bytes: a buffer load
  // zeroes every dword that crosses the end of the range, which would drop a
  // last logit sharing its dword with the end.  Rows are padded to 16-byte
  // multiples of row_stride >= vocab, so the rounded range stays in the row;
  // logits past the vocabulary are masked by index.
  const int row_bytes = (a.vocab * ESIZE + 15) / 16 * 16;
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), 0, row_bytes, 0x00020000);
  const float k = a.inv_temperature * kLog2e;
  const int nchunks = (a.vocab + E - 1) / E;

  LpState st = {kFloorMax, 0.f, 0.f};
  for (int c0 = tid; c0 < nchunks; c0 += kLpThreads * kLpUnroll) {
    uint4 u[kLpUnroll];
#pragma unroll
    for (int j = 0; j < kLpUnroll; ++j) {  // loads past the row come back as zeros (masked below)
      const u32x4_t t = __builtin_amdgcn_raw_buffer_load_b128(rsrc, (c0 + j * kLpThreads) * 16, 0, 2);
      u[j] = make_uint4(t[0], t[1], t[2], t[3]);
    }
#pragma unroll
    for (int j = 0; j < kLpUnroll; ++j) {
      const int c = c0 + j * kLpThreads;
      float x[E];
      unpack<ESIZE>(u[j], x);
      float mx = kFloorMax;
#pragma unroll
      for (int e = 0; e < E; ++e)
        if (c * E + e < a.vocab) mx = fmaxf(mx, x[e]);
      if (mx > st.m) {  // the max grows: rescale the state
        const float dm = (st.m - mx) * k;
        const float sc = __builtin_amdgcn_exp2f(dm);
        st.t = st.s > 0.f ? (st.t + dm * st.s) * sc : 0.f;
        st.s *= sc;
        st.m = mx;
      }
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const float d = (x[e] - st.m) * k;
        const float p = c * E + e < a.vocab ? __builtin_amdgcn_exp2f(d) : 0.f;
        st.s += p;
        st.t += p > 0.f ? p * d : 0.f;  // a zero-probability term adds nothing, also at -inf
      }
    }
  }
  // ---- combine: wavefront butterfly, then the wavefronts in index order ----
  for (int o = 1; o < kWaveSize; o <<= 1) {
    LpState other = {__shfl_xor(st.m, o), __shfl_xor(st.s, o), __shfl_xor(st.t, o)};
    st = (tid & o) ? lp_merge(other, st, k) : lp_merge(st, other, k);  // the same order in both lanes
  }
  const int w = tid / kWaveSize;
  if ((tid & (kWaveSize - 1)) == 0) s_state[w] = st;
  __syncthreads();
  if (tid == 0) {
    LpState r = s_state[0];
    for (int x = 1; x < kLpThreads / kWaveSize; ++x) r = lp_merge(r, s_state[x], k);
    const float log2s = __builtin_amdgcn_logf(r.s);  // log2
    const int tok = a.tokens[row];
    float lp;
    if (tok >= 0 && tok < a.vocab) {
      const char* p = base + (size_t)tok * ESIZE;
      const float raw = ESIZE == 2 ? __uint_as_float((unsigned)*reinterpret_cast<const uint16_t*>(p) << 16)
                                   : *reinterpret_cast<const float*>(p);
      lp = kLn2 * ((raw - r.m) * k - log2s);
    } else {
      lp = __builtin_nanf("");
    }
    a.logprobs[row] = lp;
    if (a.entropies) a.entropies[row] = kLn2 * (log2s - r.t / r.s);
  }
}

}  // namespace

hipError_t launch_logprob(const LogprobArgs& a, hipStream_t stream) {
  if (a.elem_bytes == 2)
    hipLaunchKernelGGL(logprob_kernel<2>, dim3(a.num_rows), dim3(kLpThreads), 0, stream, a);
  else if (a.elem_bytes == 4)
    hipLaunchKernelGGL(logprob_kernel<4>, dim3(a.num_rows), dim3(kLpThreads), 0, stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pda
