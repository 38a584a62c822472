// Token log-probabilities and entropies of one decode step's LM-head logits:
// the rollout records the log-probability of every sampled token, and the
// policy loss uses the entropy of the same distribution (Appendix C).
//
// With x_j = logits[r][j] / T over the vocabulary:
//   logprob[r] = x_tok - log sum_j e^{x_j},  entropy[r] = -sum_j p_j log p_j.
//
// Each row (250-300 KB for Llama-3 / Qwen vocabularies in bf16) is streamed
// once by one 1024-thread workgroup or -- when a batch has fewer rows than
// the GPU has compute units and the caller gives a workspace -- by `slices`
// workgroups that take equal contiguous ranges of it, with 16-byte
// non-temporal buffer loads (descriptor = the row, so no read leaves it):
// a pass is two 16-byte chunks per thread, and the next pass's loads are
// issued before a pass is folded (four loads in flight per thread; on
// MI355X 2+2 ran 1% faster than 4 loads without the overlap and 7% faster
// than 4+4).  Slice workgroups leave their states in the workspace, and a
// small second kernel merges each row's states in slice order.
//
// With k = log2(e) / T, each thread keeps an online state relative to a
// reference mk (an fp32 multiple of k, never above k times the
// largest logit it has seen):
//   s = sum 2^d,  t = sum 2^d d,  d = fma(logit, k, -mk).
// The hot loop computes no max: it folds a pass of chunks against the
// current reference, and only when that makes s exceed 2^64 (some logit
// outgrew the reference by that much, or the reference is the floor of a
// fresh state) does the thread take the pass again from its saved state,
// with the reference moved to k times the pass's largest logit.  The first
// pass starts from k times its first logit.  The fused multiply-add rounds d
// once, so a large common offset of the logits (+-30000, say) costs no
// precision, and the rounding of mk shifts every d of the state by the same
// amount, which cancels in both results below.  t is relative to mk, so
// t / s stays small and the entropy keeps its precision in fp32.  The states
// are combined over the workgroup in a fixed order (a wavefront butterfly,
// then the 16 wavefronts in index order), so results are reproducible.
// Finally
//   logprob = ln2 (fma(logit_tok, k, -mk) - log2 s),  entropy = ln2 (log2 s - t / s).
// The hot loop covers whole 16-byte chunks of the vocabulary; the one partial
// chunk at its end is handled after it, with elements past the vocabulary at
// probability 0.  -inf logits get 2^-inf = 0 and add nothing to s.  The hot
// loop leaves d unguarded in t (one instruction less per logit), so a
// workgroup whose range holds a -inf logit gets a NaN t there; it takes t
// again in a second, guarded pass over its range against its final
// reference.  A token id
// outside [0, vocab) gives NaN.  The inverse temperature must be >= 0 (the
// host checks it), so the max of the logits is the max of the scaled values.
#include "pda_internal.h"

namespace pda {
namespace {

constexpr int kLpUnroll = 2;  // 16-byte loads per thread and pass (two passes in flight)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kFloorMax = -1e30f;  // running max (raw logit units) before any finite logit
constexpr float kLpOverflow = 18446744073709551616.f;  // 2^64: s above it retakes the pass

struct LpState {
  float mk, s, t;  // reference (fp32, k times a logit), sum 2^d, sum 2^d d
};

// Merge two states (both relative to their own mk).
__device__ __forceinline__ LpState lp_merge(LpState a, LpState b) {
  const float MK = fmaxf(a.mk, b.mk);
  const float da = a.mk - MK, db = b.mk - MK;  // <= 0
  const float fa = __builtin_amdgcn_exp2f(da);
  const float fb = __builtin_amdgcn_exp2f(db);
  // sum p (d relative to MK) = sum p (d relative to mk) + (mk - MK) sum p, rescaled
  LpState r;
  r.mk = MK;
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

// The row's outputs from its final state.
template <int ESIZE, bool ENTROPY>
__device__ __forceinline__ void write_outputs(const LogprobArgs& a, int row, const LpState& r) {
  const float k = a.inv_temperature * kLog2e;
  const float log2s = __builtin_amdgcn_logf(r.s);  // log2
  const int tok = a.tokens[row];
  float lp;
  if (tok >= 0 && tok < a.vocab) {
    const char* p = static_cast<const char*>(a.logits) + ((size_t)row * a.row_stride + tok) * ESIZE;
    const float raw = ESIZE == 2 ? __uint_as_float((unsigned)*reinterpret_cast<const uint16_t*>(p) << 16)
                                 : *reinterpret_cast<const float*>(p);
    lp = kLn2 * (fmaf(raw, k, -r.mk) - log2s);
  } else {
    lp = __builtin_nanf("");
  }
  a.logprobs[row] = lp;
  if (ENTROPY) a.entropies[row] = kLn2 * (log2s - r.t / r.s);
}

// ESIZE: bytes per logit (2 = bf16, 4 = fp32).  ENTROPY: whether t (and the
// entropy) is accumulated; without it a logit costs two VALU instructions
// less, for callers that record log-probabilities only.
template <int ESIZE, bool ENTROPY>
__global__ void __launch_bounds__(kLpThreads) logprob_kernel(const LogprobArgs a) {
  constexpr int E = 16 / ESIZE;  // logits per 16-byte load
  __shared__ LpState s_state[kLpThreads / kWaveSize];
  const int S = a.slices;
  const int row = blockIdx.x / S;
  const int slice = blockIdx.x % S;
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

  LpState st = {kFloorMax * k, 0.f, 0.f};
  // Move the reference up to mk (>= st.mk) and rescale the state.
  auto rescale_to = [&](float mk) {
    const float dm = st.mk - mk;
    const float sc = __builtin_amdgcn_exp2f(dm);
    st.t = st.s > 0.f ? (st.t + dm * st.s) * sc : 0.f;
    st.s *= sc;
    st.mk = mk;
  };
  // Fold `valid` logits of a chunk against the current reference (elements
  // past the vocabulary, only in the last, partial chunk, get probability 0).
  auto fold = [&](const float (&x)[E], int valid) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      if (e < valid) {
        const float d = fmaf(x[e], k, -st.mk);
        const float p = __builtin_amdgcn_exp2f(d);
        st.s += p;
        // A -inf logit (d = -inf, p = 0) makes t NaN here; such a row's t is
        // taken again, guarded, after the combine.
        if constexpr (ENTROPY) st.t = fmaf(p, d, st.t);
      }
    }
  };
  // k times the largest of `valid` logits, floored
  auto top = [&](const float (&x)[E], int valid) {
    float mx = kFloorMax;
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (e < valid) mx = fmaxf(mx, x[e]);
    return mx * k;
  };
  auto load = [&](int c) {
    const u32x4_t t = __builtin_amdgcn_raw_buffer_load_b128(rsrc, c * 16, 0, 2);
    return make_uint4(t[0], t[1], t[2], t[3]);
  };
  const int nfull = a.vocab / E;  // whole chunks
  const int per_slice = (nfull + S - 1) / S;
  const int c_begin = min(nfull, slice * per_slice);
  const int c_end = min(nfull, c_begin + per_slice);  // this workgroup's whole chunks
  const bool last_slice = slice == S - 1;
  // Passes of kLpUnroll chunks per thread, software-pipelined: the loads of
  // the next pass are issued before this one is folded, so every thread keeps
  // loads in flight while it computes.  A chunk past the workgroup's range is
  // loaded at an offset past the descriptor, which reads nothing and returns
  // zeros (it is never folded).
  constexpr int kStride = kLpUnroll * kLpThreads;
  auto issue = [&](uint4 (&dst)[kLpUnroll], int c) {
#pragma unroll
    for (int j = 0; j < kLpUnroll; ++j) dst[j] = load(c + j * kLpThreads < c_end ? c + j * kLpThreads : 0x07ffffff);
  };
  bool first = true;  // the same in every thread that runs the loop
  uint4 u[kLpUnroll], nu[kLpUnroll];
  int c = c_begin + tid;
  if (c < c_end) issue(u, c);
  for (; c < c_end; c += kStride) {
    issue(nu, c + kStride);
    // The pass's fold at raised wave priority (the next loads are issued at
    // the normal one): a wavefront that has its data finishes its pass and
    // issues its next loads sooner (bf16 rows on MI355X 2.5% faster).
    __builtin_amdgcn_s_setprio(1);
    if (first) {  // a reference from the pass's first logit (always a whole chunk's)
      first = false;
      float x[E];
      unpack<ESIZE>(u[0], x);
      st.mk = fmaxf(st.mk, x[0] * k);
    }
    const LpState saved = st;
#pragma unroll
    for (int j = 0; j < kLpUnroll; ++j) {
      if (c + j * kLpThreads < c_end) {
        float x[E];
        unpack<ESIZE>(u[j], x);
        fold(x, E);
      }
    }
    if (st.s > kLpOverflow) {  // rare: again from the saved state, against the pass's max
      st = saved;
      float mk = st.mk;
#pragma unroll
      for (int j = 0; j < kLpUnroll; ++j) {
        if (c + j * kLpThreads < c_end) {
          float x[E];
          unpack<ESIZE>(u[j], x);
          mk = fmaxf(mk, top(x, E));
        }
      }
      if (mk > st.mk) rescale_to(mk);
#pragma unroll
      for (int j = 0; j < kLpUnroll; ++j) {
        if (c + j * kLpThreads < c_end) {
          float x[E];
          unpack<ESIZE>(u[j], x);
          fold(x, E);
        }
      }
    }
    __builtin_amdgcn_s_setprio(0);
#pragma unroll
    for (int j = 0; j < kLpUnroll; ++j) u[j] = nu[j];
  }
  // the partial chunk (the descriptor covers it), in the last slice
  const int partial_tid = (nfull - c_begin) % kLpThreads;
  const bool has_partial = last_slice && nfull * E < a.vocab;
  if (has_partial && tid == partial_tid) {
    float x[E];
    unpack<ESIZE>(load(nfull), x);
    const int valid = a.vocab - nfull * E;
    const float mk = top(x, valid);
    if (mk > st.mk) rescale_to(mk);
    fold(x, valid);
  }
  // ---- combine: wavefront butterfly, then the wavefronts in index order ----
  for (int o = 1; o < kWaveSize; o <<= 1) {
    LpState other = {__shfl_xor(st.mk, o), __shfl_xor(st.s, o), __shfl_xor(st.t, o)};
    st = (tid & o) ? lp_merge(other, st) : lp_merge(st, other);  // the same order in both lanes
  }
  const int w = tid / kWaveSize;
  if ((tid & (kWaveSize - 1)) == 0) s_state[w] = st;
  __syncthreads();
  LpState r = {0.f, 0.f, 0.f};
  __shared__ int s_redo;
  __shared__ float s_ref;
  if (w == 0) {  // the wavefronts' states in index order
    r = s_state[0];
    for (int x = 1; x < kLpThreads / kWaveSize; ++x) r = lp_merge(r, s_state[x]);
    if (ENTROPY && tid == 0) {
      s_redo = __builtin_isnan(r.t) && __builtin_isfinite(r.s);
      s_ref = r.mk;
    }
  }
  if (ENTROPY) __syncthreads();
  if (ENTROPY && s_redo) {
    // Some logit of this workgroup's range is -inf (a NaN logit would have
    // made s NaN as well): take t again against the final reference, with d
    // floored so that those logits add 0 * floor = 0.  s is unchanged (they
    // add 0 to it either way).
    __shared__ float s_tsum[kLpThreads / kWaveSize];
    const float ref = s_ref;
    float t = 0.f;
    auto fold_t = [&](const float (&x)[E], int valid) {
#pragma unroll
      for (int e = 0; e < E; ++e)
        if (e < valid) {
          const float d = fmaf(x[e], k, -ref);
          t = fmaf(__builtin_amdgcn_exp2f(d), fmaxf(d, kFloorMax), t);
        }
    };
    for (int cc = c_begin + tid; cc < c_end; cc += kLpThreads) {
      float x[E];
      unpack<ESIZE>(load(cc), x);
      fold_t(x, E);
    }
    if (has_partial && tid == partial_tid) {
      float x[E];
      unpack<ESIZE>(load(nfull), x);
      fold_t(x, a.vocab - nfull * E);
    }
    for (int o = 1; o < kWaveSize; o <<= 1) t += __shfl_xor(t, o);
    if ((tid & (kWaveSize - 1)) == 0) s_tsum[w] = t;
    __syncthreads();
    r.t = s_tsum[0];
    for (int x = 1; x < kLpThreads / kWaveSize; ++x) r.t += s_tsum[x];
  }
  if (tid == 0) {
    if (S == 1) {
      write_outputs<ESIZE, ENTROPY>(a, row, r);
    } else {  // the row's other slices: logprob_merge_kernel combines them
      float* p = a.part + ((size_t)row * S + slice) * 4;
      *reinterpret_cast<f32x4_t*>(p) = f32x4_t{r.mk, r.s, r.t, 0.f};
    }
  }
}

// Pass 2 of a row split over workgroups: one thread per row merges the
// slices' states in slice order and writes the outputs.
template <int ESIZE, bool ENTROPY>
__global__ void __launch_bounds__(kWaveSize) logprob_merge_kernel(const LogprobArgs a) {
  const int row = blockIdx.x * kWaveSize + threadIdx.x;
  if (row >= a.num_rows) return;
  const int S = a.slices;
  const f32x4_t* p = reinterpret_cast<const f32x4_t*>(a.part) + (size_t)row * S;
  f32x4_t v = p[0];
  LpState r = {v[0], v[1], v[2]};
  for (int x = 1; x < S; ++x) {
    v = p[x];
    r = lp_merge(r, LpState{v[0], v[1], v[2]});
  }
  write_outputs<ESIZE, ENTROPY>(a, row, r);
}

}  // namespace

namespace {

template <int ESIZE, bool ENTROPY>
hipError_t launch_t(const LogprobArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL((logprob_kernel<ESIZE, ENTROPY>), dim3((unsigned)a.num_rows * (unsigned)a.slices),
                     dim3(kLpThreads), 0, stream, a);
  if (a.slices > 1) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((logprob_merge_kernel<ESIZE, ENTROPY>), dim3((a.num_rows + kWaveSize - 1) / kWaveSize),
                       dim3(kWaveSize), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_logprob(const LogprobArgs& a, hipStream_t stream) {
  const bool ent = a.entropies != nullptr;
  if (a.elem_bytes == 2) return ent ? launch_t<2, true>(a, stream) : launch_t<2, false>(a, stream);
  if (a.elem_bytes == 4) return ent ? launch_t<4, true>(a, stream) : launch_t<4, false>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace pda
