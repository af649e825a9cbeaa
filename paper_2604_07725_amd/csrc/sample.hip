// Fused full-vocabulary log-softmax + Gumbel-max sampling.
//
// Pass 1: one 256-thread workgroup per (4096-entry vocab chunk, candidate).
// Each thread owns four Philox4x32-10 counters = 16 consecutive vocab entries
// read as four 16-byte loads, computes z = logit / T, the chunk-local max and
// sum of exp(z - max) (wavefront shuffle reductions, then LDS), and the best
// perturbed value z + G (ties -> lowest index).  Pass 2: one workgroup per
// candidate merges its chunks in a fixed order and writes the token id and
// log-probability z_id - logsumexp(z).
//
// Optionally (conf_k > 0) the same passes produce the per-token confidence of
// the group-confidence fitness signal (Eq. 1): c = logsumexp(x) - mean of the
// conf_k largest logits x, i.e. minus the mean of the top-conf_k
// log-probabilities under the model's own distribution (T = 1).  Pass 1 keeps
// each chunk's conf_k largest logits (per-wave extraction, then a merge of the
// four waves), pass 2 merges the chunks' lists.
//
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): 10 rounds; round r uses
// key + r * (0x9E3779B9, 0xBB67AE85); multipliers 0xD2511F53, 0xCD9E8D57.
// Counter (v >> 2, position, uid lo, uid hi), key (seed lo, seed hi), word v & 3.
// u = ((w >> 9) + 0.5) 2^-23 (exact in fp32), G = -log(-log u).
#include "common.h"
#include "kernels.h"

namespace sevo {

__device__ __forceinline__ u32x4 philox4x32_10(u32x4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint32_t lo0 = 0xD2511F53u * c.x;
    const uint32_t hi0 = __umulhi(0xD2511F53u, c.x);
    const uint32_t lo1 = 0xCD9E8D57u * c.z;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c.z);
    c = u32x4{hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0};
  }
  return c;
}

__device__ __forceinline__ float gumbel_from_bits(uint32_t w) {
  const float u = ((float)(w >> 9) + 0.5f) * 1.1920928955078125e-07f;  // 2^-23
  return -logf(-logf(u));
}

struct SamplePartial {
  float m;     // max z in the chunk
  float s;     // sum exp(z - m)
  float best;  // best perturbed value
  int idx;     // its vocab index
  float m1;    // max and sum exp of the raw logits (T = 1), for the confidence
  float s1;
};

constexpr int kConfMaxK = 32;     // largest supported top-K of the confidence
constexpr int kConfMergeNV = 24;  // list entries per lane in the chunk merge

__device__ __forceinline__ void lse_merge(float& m, float& s, float om, float os) {
  const float M = fmaxf(m, om);
  s = (m == -INFINITY ? 0.f : s * expf(m - M)) + (om == -INFINITY ? 0.f : os * expf(om - M));
  m = M;
}

// The K largest of the values a wave holds (NV per lane; -inf = empty), in
// descending order, written by lane 0 to out[0..K).  Each round takes the wave
// maximum (ties: lowest lane, then slot) and removes it from its lane.
template <int NV>
__device__ __forceinline__ void wave_topk(float (&x)[NV], int K, float* out) {
  const int lane = threadIdx.x & 63;
  for (int r = 0; r < K; ++r) {
    float bv = -INFINITY;
    int bs = 0;
#pragma unroll
    for (int e = 0; e < NV; ++e)
      if (x[e] > bv) {
        bv = x[e];
        bs = e;
      }
    int key = lane * NV + bs;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(bv, o, kWave);
      const int ok = __shfl_xor(key, o, kWave);
      if (ov > bv || (ov == bv && ok < key)) {
        bv = ov;
        key = ok;
      }
    }
    if (lane == key / NV) {
      const int slot = key - (key / NV) * NV;
#pragma unroll
      for (int e = 0; e < NV; ++e)
        if (e == slot) x[e] = -INFINITY;
    }
    if (lane == 0) out[r] = bv;
  }
}

__device__ __forceinline__ bool better(float a, int ia, float b, int ib) {
  return a > b || (a == b && ia < ib);
}

template <int NW>
__device__ __forceinline__ SamplePartial block_merge(SamplePartial p, SamplePartial* red) {
  // wave level
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float om = __shfl_xor(p.m, o, kWave);
    const float os = __shfl_xor(p.s, o, kWave);
    const float ob = __shfl_xor(p.best, o, kWave);
    const int oi = __shfl_xor(p.idx, o, kWave);
    const float om1 = __shfl_xor(p.m1, o, kWave);
    const float os1 = __shfl_xor(p.s1, o, kWave);
    lse_merge(p.m, p.s, om, os);
    lse_merge(p.m1, p.s1, om1, os1);
    if (better(ob, oi, p.best, p.idx)) {
      p.best = ob;
      p.idx = oi;
    }
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = p;
  __syncthreads();
  SamplePartial r = red[0];
#pragma unroll
  for (int k = 1; k < NW; ++k) {
    const SamplePartial o = red[k];
    lse_merge(r.m, r.s, o.m, o.s);
    lse_merge(r.m1, r.s1, o.m1, o.s1);
    if (better(o.best, o.idx, r.best, r.idx)) {
      r.best = o.best;
      r.idx = o.idx;
    }
  }
  return r;
}

__global__ __launch_bounds__(256) void sample_partial_kernel(
    const float* __restrict__ logits, int vocab, int64_t ld, float temp, uint64_t seed,
    const uint64_t* __restrict__ uid, const int32_t* __restrict__ positions,
    SamplePartial* __restrict__ part, int conf_k, float* __restrict__ topk) {
  __shared__ SamplePartial red[4];
  __shared__ float wtop[4][kConfMaxK];
  const int chunk = blockIdx.x;
  const int i = blockIdx.y;
  const float* row = logits + (size_t)i * ld;
  const bool greedy = temp == 0.f;
  const bool unit_t = temp == 1.f;
  const uint64_t cu = uid[i];
  const uint32_t pos = (uint32_t)positions[i];
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  float z[16], raw[16];
  float best = -INFINITY;
  int bidx = 0x7FFFFFFF;
  float m = -INFINITY;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int q4 = chunk * (kSampleChunk / 4) + r * 256 + threadIdx.x;  // Philox counter word 0
    const int v0 = q4 * 4;
    float4 lv;
    if (v0 + 3 < vocab) {
      lv = *reinterpret_cast<const float4*>(row + v0);
    } else {
      lv.x = v0 + 0 < vocab ? row[v0 + 0] : -INFINITY;
      lv.y = v0 + 1 < vocab ? row[v0 + 1] : -INFINITY;
      lv.z = v0 + 2 < vocab ? row[v0 + 2] : -INFINITY;
      lv.w = v0 + 3 < vocab ? row[v0 + 3] : -INFINITY;
    }
    float zz[4] = {lv.x, lv.y, lv.z, lv.w};
    raw[r * 4 + 0] = lv.x;
    raw[r * 4 + 1] = lv.y;
    raw[r * 4 + 2] = lv.z;
    raw[r * 4 + 3] = lv.w;
    if (!greedy && !unit_t) {
#pragma unroll
      for (int e = 0; e < 4; ++e) zz[e] = zz[e] / temp;
    }
    float g[4] = {0.f, 0.f, 0.f, 0.f};
    if (!greedy && v0 < vocab) {
      const u32x4 w = philox4x32_10(u32x4{(uint32_t)q4, pos, (uint32_t)cu, (uint32_t)(cu >> 32)},
                                    k0, k1);
      g[0] = gumbel_from_bits(w.x);
      g[1] = gumbel_from_bits(w.y);
      g[2] = gumbel_from_bits(w.z);
      g[3] = gumbel_from_bits(w.w);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      z[r * 4 + e] = zz[e];
      m = fmaxf(m, zz[e]);
      const int v = v0 + e;
      if (v < vocab) {
        const float pv = zz[e] + g[e];
        if (pv > best) {  // ascending v within a thread: strict > keeps the lowest index
          best = pv;
          bidx = v;
        }
      }
    }
  }
  // greedy sampling reports log-probs under T = 1, and z = logits there
  float s = 0.f;
  if (m != -INFINITY) {
#pragma unroll
    for (int e = 0; e < 16; ++e) s += (z[e] == -INFINITY) ? 0.f : expf(z[e] - m);
  }
  // statistics of the raw logits (T = 1) for the confidence; equal to the
  // above when z is the raw logit
  float m1 = m, s1 = s;
  if (conf_k > 0 && !greedy && !unit_t) {
    m1 = -INFINITY;
#pragma unroll
    for (int e = 0; e < 16; ++e) m1 = fmaxf(m1, raw[e]);
    s1 = 0.f;
    if (m1 != -INFINITY) {
#pragma unroll
      for (int e = 0; e < 16; ++e) s1 += (raw[e] == -INFINITY) ? 0.f : expf(raw[e] - m1);
    }
  }
  SamplePartial p{m, s, best, bidx, m1, s1};
  p = block_merge<4>(p, red);
  if (threadIdx.x == 0) part[(size_t)i * gridDim.x + chunk] = p;
  if (conf_k > 0) {
    // the chunk's conf_k largest raw logits: per wave, then merged by wave 0
    const int wave = threadIdx.x >> 6;
    wave_topk<16>(raw, conf_k, wtop[wave]);
    __syncthreads();
    if (wave == 0) {
      const int lane = threadIdx.x & 63;
      float x2[2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int q = lane * 2 + e;  // entry q of the 4 lists of conf_k values
        const int w = q / kConfMaxK, r = q - w * kConfMaxK;
        x2[e] = (w < 4 && r < conf_k) ? wtop[w][r] : -INFINITY;
      }
      wave_topk<2>(x2, conf_k, topk + ((size_t)i * gridDim.x + chunk) * kConfMaxK);
    }
  }
}

__global__ __launch_bounds__(256) void sample_final_kernel(
    const SamplePartial* __restrict__ part, int nchunks, const float* __restrict__ logits,
    int64_t ld, float temp, int32_t* __restrict__ out_tokens, float* __restrict__ out_lp,
    int conf_k, const float* __restrict__ topk, float* __restrict__ out_conf,
    float* __restrict__ conf_sum) {
  __shared__ SamplePartial red[4];
  __shared__ float wtop[4][kConfMaxK];
  const int i = blockIdx.x;
  SamplePartial p{-INFINITY, 0.f, -INFINITY, 0x7FFFFFFF, -INFINITY, 0.f};
  for (int c = threadIdx.x; c < nchunks; c += 256) {
    const SamplePartial o = part[(size_t)i * nchunks + c];
    lse_merge(p.m, p.s, o.m, o.s);
    lse_merge(p.m1, p.s1, o.m1, o.s1);
    if (better(o.best, o.idx, p.best, p.idx)) {
      p.best = o.best;
      p.idx = o.idx;
    }
  }
  p = block_merge<4>(p, red);
  if (threadIdx.x == 0) {
    const int id = p.idx;
    float zid = logits[(size_t)i * ld + id];
    if (temp != 0.f && temp != 1.f) zid = zid / temp;
    out_tokens[i] = id;
    out_lp[i] = zid - (p.m + logf(p.s));
  }
  if (conf_k > 0) {
    // merge the chunks' lists: wave w takes a contiguous quarter of them, then
    // wave 0 merges the four results (host checks nchunks * conf_k fits)
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int total = nchunks * conf_k;
    const int per = (total + 3) / 4;
    const float* src = topk + (size_t)i * nchunks * kConfMaxK;
    float x[kConfMergeNV];
#pragma unroll
    for (int e = 0; e < kConfMergeNV; ++e) {
      const int q = wave * per + lane * kConfMergeNV + e;  // entry of the flattened lists
      const bool ok = lane * kConfMergeNV + e < per && q < total;
      const int c = ok ? q / conf_k : 0;
      x[e] = ok ? src[(size_t)c * kConfMaxK + (q - c * conf_k)] : -INFINITY;
    }
    wave_topk<kConfMergeNV>(x, conf_k, wtop[wave]);
    __syncthreads();
    if (wave == 0) {
      float x2[2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int q = lane * 2 + e;
        const int w = q / kConfMaxK, r = q - w * kConfMaxK;
        x2[e] = (w < 4 && r < conf_k) ? wtop[w][r] : -INFINITY;
      }
      __shared__ float top[kConfMaxK];
      wave_topk<2>(x2, conf_k, top);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      if (lane == 0) {
        float sum = 0.f;
        for (int r = 0; r < conf_k; ++r) sum += top[r];
        const float c = (p.m1 + logf(p.s1)) - sum / (float)conf_k;
        if (out_conf) out_conf[i] = c;
        if (conf_sum) conf_sum[i] += c;
      }
    }
  }
}

// GC(g) = (1/K) sum over the group's candidates of conf_sum / token count (Eq. 2)
__global__ __launch_bounds__(256) void group_confidence_kernel(
    const float* __restrict__ conf_sum, const int32_t* __restrict__ counts,
    const int32_t* __restrict__ groups, int n_groups, int K, float* __restrict__ out) {
  const int g = blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= n_groups) return;
  float a = 0.f;
  for (int k = 0; k < K; ++k) {
    const int c = groups[(size_t)g * K + k];
    a += conf_sum[c] / (float)counts[c];
  }
  out[g] = a / (float)K;
}

static size_t partial_bytes(int n, int nchunks) {
  return ((size_t)n * nchunks * sizeof(SamplePartial) + 255) / 256 * 256;
}

size_t sample_workspace_bytes(int n, int vocab) {
  const int nchunks = (vocab + kSampleChunk - 1) / kSampleChunk;
  return partial_bytes(n, nchunks) + (size_t)n * nchunks * kConfMaxK * sizeof(float);
}

bool sample_conf_supported(int vocab, int conf_k) {
  const int nchunks = (vocab + kSampleChunk - 1) / kSampleChunk;
  return conf_k >= 0 && conf_k <= kConfMaxK && conf_k <= vocab &&
         (size_t)nchunks * conf_k <= (size_t)4 * kWave * kConfMergeNV;
}

hipError_t launch_logprob_sample(const float* logits, int n, int vocab, int64_t ld, float temp,
                                 uint64_t seed, const uint64_t* uid, const int32_t* positions,
                                 int32_t* out_tokens, float* out_lp, float* workspace,
                                 int conf_k, float* out_conf, float* conf_sum, hipStream_t st) {
  if (n == 0) return hipSuccess;
  const int nchunks = (vocab + kSampleChunk - 1) / kSampleChunk;
  SamplePartial* part = reinterpret_cast<SamplePartial*>(workspace);
  float* topk = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) +
                                         partial_bytes(n, nchunks));
  hipLaunchKernelGGL(sample_partial_kernel, dim3(nchunks, n), dim3(256), 0, st, logits, vocab, ld,
                     temp, seed, uid, positions, part, conf_k, topk);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sample_final_kernel, dim3(n), dim3(256), 0, st, part, nchunks, logits, ld,
                     temp, out_tokens, out_lp, conf_k, topk, out_conf, conf_sum);
  return hipGetLastError();
}

hipError_t launch_group_confidence(const float* conf_sum, const int32_t* counts,
                                   const int32_t* groups, int n_groups, int K, float* out,
                                   hipStream_t st) {
  if (n_groups == 0) return hipSuccess;
  hipLaunchKernelGGL(group_confidence_kernel, dim3((n_groups + 255) / 256), dim3(256), 0, st,
                     conf_sum, counts, groups, n_groups, K, out);
  return hipGetLastError();
}

}  // namespace sevo
