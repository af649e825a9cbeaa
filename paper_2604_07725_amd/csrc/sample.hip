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
};

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
    const float M = fmaxf(p.m, om);
    const float s = (p.m == -INFINITY ? 0.f : p.s * expf(p.m - M)) +
                    (om == -INFINITY ? 0.f : os * expf(om - M));
    p.m = M;
    p.s = s;
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
    const float M = fmaxf(r.m, o.m);
    r.s = (r.m == -INFINITY ? 0.f : r.s * expf(r.m - M)) +
          (o.m == -INFINITY ? 0.f : o.s * expf(o.m - M));
    r.m = M;
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
    SamplePartial* __restrict__ part) {
  __shared__ SamplePartial red[4];
  const int chunk = blockIdx.x;
  const int i = blockIdx.y;
  const float* row = logits + (size_t)i * ld;
  const bool greedy = temp == 0.f;
  const bool unit_t = temp == 1.f;
  const uint64_t cu = uid[i];
  const uint32_t pos = (uint32_t)positions[i];
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  float z[16];
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
  SamplePartial p{m, s, best, bidx};
  p = block_merge<4>(p, red);
  if (threadIdx.x == 0) part[(size_t)i * gridDim.x + chunk] = p;
}

__global__ __launch_bounds__(256) void sample_final_kernel(
    const SamplePartial* __restrict__ part, int nchunks, const float* __restrict__ logits,
    int64_t ld, float temp, int32_t* __restrict__ out_tokens, float* __restrict__ out_lp) {
  __shared__ SamplePartial red[4];
  const int i = blockIdx.x;
  SamplePartial p{-INFINITY, 0.f, -INFINITY, 0x7FFFFFFF};
  for (int c = threadIdx.x; c < nchunks; c += 256) {
    const SamplePartial o = part[(size_t)i * nchunks + c];
    const float M = fmaxf(p.m, o.m);
    p.s = (p.m == -INFINITY ? 0.f : p.s * expf(p.m - M)) +
          (o.m == -INFINITY ? 0.f : o.s * expf(o.m - M));
    p.m = M;
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
}

size_t sample_workspace_bytes(int n, int vocab) {
  const int nchunks = (vocab + kSampleChunk - 1) / kSampleChunk;
  return (size_t)n * nchunks * sizeof(SamplePartial);
}

hipError_t launch_logprob_sample(const float* logits, int n, int vocab, int64_t ld, float temp,
                                 uint64_t seed, const uint64_t* uid, const int32_t* positions,
                                 int32_t* out_tokens, float* out_lp, float* workspace,
                                 hipStream_t st) {
  if (n == 0) return hipSuccess;
  const int nchunks = (vocab + kSampleChunk - 1) / kSampleChunk;
  SamplePartial* part = reinterpret_cast<SamplePartial*>(workspace);
  hipLaunchKernelGGL(sample_partial_kernel, dim3(nchunks, n), dim3(256), 0, st, logits, vocab, ld,
                     temp, seed, uid, positions, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sample_final_kernel, dim3(n), dim3(256), 0, st, part, nchunks, logits, ld,
                     temp, out_tokens, out_lp);
  return hipGetLastError();
}

}  // namespace sevo
