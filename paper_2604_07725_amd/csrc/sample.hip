// Fused full-vocabulary log-softmax + Gumbel-max sampling.
//
// Pass 1: one 256-thread workgroup per (4096-entry vocab chunk, candidate).
// Thread t owns the 4-entry groups 1024 r + 4 t (r < 4) of the chunk, each one
// Philox4x32-10 counter and one 16-byte load; it computes z = logit / T, the
// chunk-local max and sum of exp(z - max) (wavefront shuffle reductions, then
// LDS), and the best perturbed value z + G (ties -> lowest index).  The
// temperature mode (T = 0, T = 1, other) is a template parameter, so greedy
// sampling carries no noise or division code.  Pass 2: one workgroup per
// candidate merges its chunks in a fixed order and writes the token id and
// log-probability z_id - logsumexp(z).
//
// Optionally (conf_k > 0) the same passes produce the per-token confidence of
// the group-confidence fitness signal (Eq. 1): c = logsumexp(x) - mean of the
// conf_k largest logits x, i.e. minus the mean of the top-conf_k
// log-probabilities under the model's own distribution (T = 1).  Pass 1 keeps
// each chunk's conf_k largest logits (per wave by a threshold and a bitonic
// sort, then a bitonic merge of the four waves' lists), pass 2 merges the
// chunks' lists the same way.
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

constexpr float kLog2e = 1.4426950408889634f;

// e^d for d <= 0 (or -inf) on the hardware exp2: one rounding of d log2(e),
// then v_exp_f32 (results below 2^-126 may flush to zero; they only ever add
// to sums whose largest term is 1)
__device__ __forceinline__ float exp_le0(float d) { return __builtin_amdgcn_exp2f(d * kLog2e); }

__device__ __forceinline__ void lse_merge(float& m, float& s, float om, float os) {
  const float M = fmaxf(m, om);
  s = (m == -INFINITY ? 0.f : s * exp_le0(m - M)) + (om == -INFINITY ? 0.f : os * exp_le0(om - M));
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

// Descending bitonic sort of one value per lane across the wave (21
// compare-exchange steps; values only).
__device__ __forceinline__ float wave_sort_desc(float v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int k = 2; k <= 64; k <<= 1)
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      const float o = __shfl_xor(v, j, kWave);
      v = (((lane & k) == 0) == ((lane & j) == 0)) ? fmaxf(v, o) : fminf(v, o);
    }
  return v;
}

// Descending sort of a bitonic sequence held one value per lane (6 steps).
__device__ __forceinline__ float wave_merge_desc(float v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 32; j > 0; j >>= 1) {
    const float o = __shfl_xor(v, j, kWave);
    v = (lane & j) == 0 ? fmaxf(v, o) : fminf(v, o);
  }
  return v;
}

// The same result as wave_topk (the K <= 32 largest values, descending, in
// out[0..K)), written by lanes 0..K-1, found by thresholding: L = the K-th
// largest of the 64 lane maxima is a lower bound of the K-th largest value
// (the K largest lane maxima are K values >= L), so the values >= L contain
// the top K.  When there are at most 64 of them (the common case), they are
// compacted into cand (64 floats of LDS) with ballots and sorted across the
// wave; otherwise (many equal values, or fewer than K finite ones) the wave
// falls back to wave_topk.  NaN is never taken, as in wave_topk.
template <int NV>
__device__ __forceinline__ void wave_topk_fast(float (&x)[NV], int K, float* out, float* cand) {
  const int lane = threadIdx.x & 63;
  float lm = -INFINITY;
#pragma unroll
  for (int e = 0; e < NV; ++e) lm = fmaxf(lm, x[e]);
  const float L = __shfl(wave_sort_desc(lm), K - 1, kWave);
  const uint64_t below = (1ull << lane) - 1ull;
  int n = 0;
#pragma unroll
  for (int e = 0; e < NV; ++e) {
    const bool c = x[e] >= L;
    const uint64_t m = __ballot(c);
    const int pos = n + __popcll(m & below);
    if (c && pos < kWave) cand[pos] = x[e];
    n += __popcll(m);
  }
  if (n <= kWave) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const float v = wave_sort_desc(lane < n ? cand[lane] : -INFINITY);
    if (lane < K) out[lane] = v;
  } else {
    wave_topk<NV>(x, K, out);
  }
}

// Merges four descending lists of K <= 32 values (list w at lists[w * 32])
// into their K largest, descending, returned in lanes 0..K-1 (one wave).
__device__ __forceinline__ float merge4_desc(const float* lists, int K) {
  const int lane = threadIdx.x & 63;
  auto get = [&](int w, int r) { return r < K ? lists[w * kConfMaxK + r] : -INFINITY; };
  // list 0 descending then list 1 ascending: a bitonic sequence
  const float a = wave_merge_desc(lane < 32 ? get(0, lane) : get(1, 63 - lane));
  const float b = wave_merge_desc(lane < 32 ? get(2, lane) : get(3, 63 - lane));
  const float br = __shfl(b, 63 - lane, kWave);  // lanes 32..63: b[31..0], ascending
  return wave_merge_desc(lane < 32 ? a : br);
}

__device__ __forceinline__ bool better(float a, int ia, float b, int ib) {
  return a > b || (a == b && ia < ib);
}

// RAW: the raw-logit statistics (m1, s1) differ from z's and are merged too;
// otherwise they are set equal to the merged (m, s)
template <int NW, bool RAW = true>
__device__ __forceinline__ SamplePartial block_merge(SamplePartial p, SamplePartial* red) {
  // wave level
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float om = __shfl_xor(p.m, o, kWave);
    const float os = __shfl_xor(p.s, o, kWave);
    const float ob = __shfl_xor(p.best, o, kWave);
    const int oi = __shfl_xor(p.idx, o, kWave);
    lse_merge(p.m, p.s, om, os);
    if constexpr (RAW) {
      const float om1 = __shfl_xor(p.m1, o, kWave);
      const float os1 = __shfl_xor(p.s1, o, kWave);
      lse_merge(p.m1, p.s1, om1, os1);
    }
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
    if constexpr (RAW) lse_merge(r.m1, r.s1, o.m1, o.s1);
    if (better(o.best, o.idx, r.best, r.idx)) {
      r.best = o.best;
      r.idx = o.idx;
    }
  }
  if constexpr (!RAW) {
    r.m1 = r.m;
    r.s1 = r.s;
  }
  return r;
}

// Pass 1.  MODE 0: T = 0 (greedy, no noise, z = x); 1: T = 1 (z = x); 2: any
// other T (z = x / T).  CONF: also the chunk's conf_k largest raw logits.
template <int MODE, bool CONF>
__global__ __launch_bounds__(256) void sample_partial_kernel(
    const float* __restrict__ logits, int vocab, int64_t ld, float temp, uint64_t seed,
    const uint64_t* __restrict__ uid, const int32_t* __restrict__ positions,
    SamplePartial* __restrict__ part, int conf_k, float* __restrict__ topk) {
  __shared__ SamplePartial red[4];
  __shared__ float wtop[4][kConfMaxK];
  __shared__ float cand[4][kWave];
  const int chunk = blockIdx.x;
  const int i = blockIdx.y;
  const float* row = logits + (size_t)i * ld;
  float raw[16];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int v0 = (chunk * (kSampleChunk / 4) + r * 256 + threadIdx.x) * 4;
    float4 lv;
    if (v0 + 3 < vocab) {
      lv = *reinterpret_cast<const float4*>(row + v0);
    } else {
      lv.x = v0 + 0 < vocab ? row[v0 + 0] : -INFINITY;
      lv.y = v0 + 1 < vocab ? row[v0 + 1] : -INFINITY;
      lv.z = v0 + 2 < vocab ? row[v0 + 2] : -INFINITY;
      lv.w = v0 + 3 < vocab ? row[v0 + 3] : -INFINITY;
    }
    raw[4 * r + 0] = lv.x;
    raw[4 * r + 1] = lv.y;
    raw[4 * r + 2] = lv.z;
    raw[4 * r + 3] = lv.w;
  }
  float z[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) z[e] = MODE == 2 ? raw[e] / temp : raw[e];
  // the best perturbed value z + G (greedy: G = 0); v ascends within a
  // thread, so the strict > keeps the lowest index of a tie
  float best = -INFINITY;
  int bidx = 0x7FFFFFFF;
  uint64_t cu = 0;
  uint32_t pos = 0;
  if constexpr (MODE != 0) {
    cu = uid[i];
    pos = (uint32_t)positions[i];
  }
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int q4 = chunk * (kSampleChunk / 4) + r * 256 + threadIdx.x;  // Philox counter word 0
    const int v0 = q4 * 4;
    float g[4] = {0.f, 0.f, 0.f, 0.f};
    if constexpr (MODE != 0) {
      if (v0 < vocab) {
        const u32x4 w = philox4x32_10(
            u32x4{(uint32_t)q4, pos, (uint32_t)cu, (uint32_t)(cu >> 32)}, k0, k1);
        g[0] = gumbel_from_bits(w.x);
        g[1] = gumbel_from_bits(w.y);
        g[2] = gumbel_from_bits(w.z);
        g[3] = gumbel_from_bits(w.w);
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float pv = z[4 * r + e] + g[e];
      if (v0 + e < vocab && pv > best) {
        best = pv;
        bidx = v0 + e;
      }
    }
  }
  // max and sum of exp(z - max); for MODE 2 with the confidence also those
  // of the raw logits (T = 1), else they are z's
  auto lse16 = [](const float (&x)[16], float& m, float& s) {
    m = -INFINITY;
#pragma unroll
    for (int e = 0; e < 16; ++e) m = fmaxf(m, x[e]);
    s = 0.f;
    if (m != -INFINITY) {
#pragma unroll
      for (int e = 0; e < 16; ++e) s += exp_le0(x[e] - m);  // exp(-inf) = 0
    }
  };
  constexpr bool kRaw = MODE == 2 && CONF;
  SamplePartial p{-INFINITY, 0.f, best, bidx, -INFINITY, 0.f};
  lse16(z, p.m, p.s);
  if constexpr (kRaw) lse16(raw, p.m1, p.s1);
  p = block_merge<4, kRaw>(p, red);
  if (threadIdx.x == 0) part[(size_t)i * gridDim.x + chunk] = p;
  if constexpr (CONF) {
    // the chunk's conf_k largest raw logits: per wave, then merged by wave 0
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    wave_topk_fast<16>(raw, conf_k, wtop[wave], cand[wave]);
    __syncthreads();
    if (wave == 0) {
      const float v = merge4_desc(&wtop[0][0], conf_k);
      if (lane < conf_k) topk[((size_t)i * gridDim.x + chunk) * kConfMaxK + lane] = v;
    }
  }
}

__global__ __launch_bounds__(256) void sample_final_kernel(
    const SamplePartial* __restrict__ part, int nchunks, const float* __restrict__ logits,
    int vocab, int64_t ld, float temp, int32_t* __restrict__ out_tokens, float* __restrict__ out_lp,
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
    if (id < 0 || id >= vocab) {
      // no perturbed value compared greater than -inf (every logit NaN): no
      // token, and the logits are not read at the missing index
      out_tokens[i] = -1;
      out_lp[i] = __builtin_nanf("");
    } else {
      float zid = logits[(size_t)i * ld + id];
      if (temp != 0.f && temp != 1.f) zid = zid / temp;
      out_tokens[i] = id;
      out_lp[i] = zid - (p.m + logf(p.s));
    }
  }
  if (conf_k > 0) {
    // merge the chunks' lists: wave w takes a contiguous quarter of them (entry
    // wave * per + 64 e + lane in lane, slot e), then wave 0 merges the four
    // results (host checks nchunks * conf_k fits)
    __shared__ float cand[4][kWave];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int total = nchunks * conf_k;
    const int per = (total + 3) / 4;
    const float* src = topk + (size_t)i * nchunks * kConfMaxK;
    float x[kConfMergeNV];
#pragma unroll
    for (int e = 0; e < kConfMergeNV; ++e) {
      const int q = wave * per + e * kWave + lane;  // entry of the flattened lists
      const bool ok = e * kWave + lane < per && q < total;
      const int c = ok ? q / conf_k : 0;
      x[e] = ok ? src[(size_t)c * kConfMaxK + (q - c * conf_k)] : -INFINITY;
    }
    wave_topk_fast<kConfMergeNV>(x, conf_k, wtop[wave], cand[wave]);
    __syncthreads();
    if (wave == 0) {
      __shared__ float top[kConfMaxK];
      const float v = merge4_desc(&wtop[0][0], conf_k);
      if (lane < conf_k) top[lane] = v;
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

// ---- truncated sampling (top-k, then min-p and top-p inside the top-k set)
//
// The kept set is the top_k logits in (value desc, vocab index asc) order --
// temperature does not change it.  With z = logit / T over that set, min-p
// keeps z_j >= z_0 + log(min_p); top-p keeps, in list order, the entries whose
// preceding cumulative probability (renormalised over the min-p set) is below
// top_p.  The token is the Gumbel-max over the kept entries (same Philox noise
// as the full sampler), lp = z_id - logsumexp(kept z).  T = 0: the first entry,
// with the truncation and lp evaluated at T = 1.
__device__ __forceinline__ bool pair_before(float a, int ia, float b, int ib) {
  return a > b || (a == b && ia < ib);
}

// The K first (value, index) pairs of a wave in pair_before order (NV per
// lane; empty = (-inf, INT_MAX)), written by lane 0 to out_v / out_i.
template <int NV>
__device__ __forceinline__ void wave_topk_pairs(float (&x)[NV], int (&xi)[NV], int K, float* out_v,
                                                int* out_i) {
  const int lane = threadIdx.x & 63;
  for (int r = 0; r < K; ++r) {
    float bv = -INFINITY;
    int bi = 0x7FFFFFFF;
#pragma unroll
    for (int e = 0; e < NV; ++e)
      if (pair_before(x[e], xi[e], bv, bi)) {
        bv = x[e];
        bi = xi[e];
      }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(bv, o, kWave);
      const int oi = __shfl_xor(bi, o, kWave);
      if (pair_before(ov, oi, bv, bi)) {
        bv = ov;
        bi = oi;
      }
    }
    // vocab indices are unique: exactly one slot holds a real winner
#pragma unroll
    for (int e = 0; e < NV; ++e)
      if (xi[e] == bi && x[e] == bv) {
        x[e] = -INFINITY;
        xi[e] = 0x7FFFFFFF;
      }
    if (lane == 0) {
      out_v[r] = bv;
      out_i[r] = bi;
    }
  }
}

__global__ __launch_bounds__(256) void sample_trunc_partial_kernel(
    const float* __restrict__ logits, int vocab, int64_t ld, int L, SamplePartial* __restrict__ part,
    float* __restrict__ topv, int* __restrict__ topi) {
  __shared__ SamplePartial red[4];
  __shared__ float wv[4][kConfMaxK];
  __shared__ int wi[4][kConfMaxK];
  const int chunk = blockIdx.x;
  const int i = blockIdx.y;
  const float* row = logits + (size_t)i * ld;
  float x[16];
  int xi[16];
  float m1 = -INFINITY;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int v0 = (chunk * (kSampleChunk / 4) + r * 256 + threadIdx.x) * 4;
    float4 lv;
    if (v0 + 3 < vocab) {
      lv = *reinterpret_cast<const float4*>(row + v0);
    } else {
      lv.x = v0 + 0 < vocab ? row[v0 + 0] : -INFINITY;
      lv.y = v0 + 1 < vocab ? row[v0 + 1] : -INFINITY;
      lv.z = v0 + 2 < vocab ? row[v0 + 2] : -INFINITY;
      lv.w = v0 + 3 < vocab ? row[v0 + 3] : -INFINITY;
    }
    const float vals[4] = {lv.x, lv.y, lv.z, lv.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[r * 4 + e] = vals[e];
      xi[r * 4 + e] = v0 + e < vocab ? v0 + e : 0x7FFFFFFF;
      m1 = fmaxf(m1, vals[e]);
    }
  }
  float s1 = 0.f;
  if (m1 != -INFINITY) {
#pragma unroll
    for (int e = 0; e < 16; ++e) s1 += (x[e] == -INFINITY) ? 0.f : expf(x[e] - m1);
  }
  SamplePartial p{m1, s1, -INFINITY, 0x7FFFFFFF, m1, s1};
  p = block_merge<4>(p, red);
  if (threadIdx.x == 0) part[(size_t)i * gridDim.x + chunk] = p;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  wave_topk_pairs<16>(x, xi, L, wv[wave], wi[wave]);
  __syncthreads();
  if (wave == 0) {
    float x2[2];
    int i2[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int q = lane * 2 + e;
      const int w = q / kConfMaxK, r = q - w * kConfMaxK;
      const bool ok = w < 4 && r < L;
      x2[e] = ok ? wv[w][r] : -INFINITY;
      i2[e] = ok ? wi[w][r] : 0x7FFFFFFF;
    }
    const size_t o = ((size_t)i * gridDim.x + chunk) * kConfMaxK;
    wave_topk_pairs<2>(x2, i2, L, topv + o, topi + o);
  }
}

__global__ __launch_bounds__(256) void sample_trunc_final_kernel(
    const SamplePartial* __restrict__ part, int nchunks, int L, const float* __restrict__ topv,
    const int* __restrict__ topi, float temp, int top_k, float top_p, float min_p, uint64_t seed,
    const uint64_t* __restrict__ uid, const int32_t* __restrict__ positions,
    int32_t* __restrict__ out_tokens, float* __restrict__ out_lp, int conf_k,
    float* __restrict__ out_conf, float* __restrict__ conf_sum) {
  __shared__ SamplePartial red[4];
  __shared__ float wv[4][kConfMaxK];
  __shared__ int wi[4][kConfMaxK];
  __shared__ float fv[kConfMaxK];
  __shared__ int fi[kConfMaxK];
  __shared__ int keep[kConfMaxK];
  const int i = blockIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  // logsumexp of the raw logits (confidence)
  SamplePartial p{-INFINITY, 0.f, -INFINITY, 0x7FFFFFFF, -INFINITY, 0.f};
  for (int c = threadIdx.x; c < nchunks; c += 256) {
    const SamplePartial o = part[(size_t)i * nchunks + c];
    lse_merge(p.m1, p.s1, o.m1, o.s1);
  }
  p.m = p.m1;
  p.s = p.s1;
  p = block_merge<4>(p, red);
  // merge the chunks' lists: a quarter per wave, then wave 0 merges the four
  const int total = nchunks * L;
  const int per = (total + 3) / 4;
  const size_t base = (size_t)i * nchunks * kConfMaxK;
  float x[kConfMergeNV];
  int xi[kConfMergeNV];
#pragma unroll
  for (int e = 0; e < kConfMergeNV; ++e) {
    const int q = wave * per + lane * kConfMergeNV + e;
    const bool ok = lane * kConfMergeNV + e < per && q < total;
    const int c = ok ? q / L : 0;
    x[e] = ok ? topv[base + (size_t)c * kConfMaxK + (q - c * L)] : -INFINITY;
    xi[e] = ok ? topi[base + (size_t)c * kConfMaxK + (q - c * L)] : 0x7FFFFFFF;
  }
  wave_topk_pairs<kConfMergeNV>(x, xi, L, wv[wave], wi[wave]);
  __syncthreads();
  if (wave != 0) return;
  {
    float x2[2];
    int i2[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int q = lane * 2 + e;
      const int w = q / kConfMaxK, r = q - w * kConfMaxK;
      const bool ok = w < 4 && r < L;
      x2[e] = ok ? wv[w][r] : -INFINITY;
      i2[e] = ok ? wi[w][r] : 0x7FFFFFFF;
    }
    wave_topk_pairs<2>(x2, i2, L, fv, fi);
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const float tdiv = temp == 0.f ? 1.f : temp;  // T = 0: truncation and lp at T = 1
  if (lane == 0) {
    // min-p, then top-p in list order over the renormalised min-p set
    const float z0 = fv[0] / tdiv;
    float tot = 0.f;
    for (int j = 0; j < top_k; ++j) {
      const float d = fv[j] / tdiv - z0;
      const bool k = !(min_p > 0.f) || d >= logf(min_p);
      keep[j] = k;
      if (k) tot += expf(d);
    }
    if (top_p < 1.f) {
      float cum = 0.f;
      for (int j = 0; j < top_k; ++j) {
        if (!keep[j]) continue;
        if (!(cum < top_p * tot)) keep[j] = 0;
        else cum += expf(fv[j] / tdiv - z0);
      }
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  // Gumbel-max over the kept entries (lane j holds entry j)
  float pv = -INFINITY, ez = 0.f;
  int pid = 0x7FFFFFFF;
  if (lane < top_k && keep[lane]) {
    const int v = fi[lane];
    const float z = fv[lane] / tdiv;
    ez = expf(z - fv[0] / tdiv);
    float g = 0.f;
    if (temp != 0.f) {
      const uint64_t cu = uid[i];
      const u32x4 w = philox4x32_10(
          u32x4{(uint32_t)(v >> 2), (uint32_t)positions[i], (uint32_t)cu, (uint32_t)(cu >> 32)},
          (uint32_t)seed, (uint32_t)(seed >> 32));
      const uint32_t word = (v & 3) == 0 ? w.x : (v & 3) == 1 ? w.y : (v & 3) == 2 ? w.z : w.w;
      g = gumbel_from_bits(word);
    }
    pv = z + g;
    pid = v;
  }
  float zme = (lane < top_k && keep[lane]) ? fv[lane] / tdiv : -INFINITY;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(pv, o, kWave);
    const int oi = __shfl_xor(pid, o, kWave);
    const float oz = __shfl_xor(zme, o, kWave);
    if (pair_before(ov, oi, pv, pid)) {
      pv = ov;
      pid = oi;
      zme = oz;
    }
    ez += __shfl_xor(ez, o, kWave);
  }
  if (lane == 0) {
    const bool found = pid >= 0 && pid != 0x7FFFFFFF;   // a kept entry won
    out_tokens[i] = found ? pid : -1;
    out_lp[i] = found ? zme - (fv[0] / tdiv + logf(ez)) : __builtin_nanf("");
    if (conf_k > 0) {
      float sum = 0.f;
      for (int r = 0; r < conf_k; ++r) sum += fv[r];
      const float c = (p.m1 + logf(p.s1)) - sum / (float)conf_k;
      if (out_conf) out_conf[i] = c;
      if (conf_sum) conf_sum[i] += c;
    }
  }
}

static size_t partial_bytes(int n, int nchunks) {
  return ((size_t)n * nchunks * sizeof(SamplePartial) + 255) / 256 * 256;
}

static size_t list_bytes(int n, int nchunks) {
  return ((size_t)n * nchunks * kConfMaxK * sizeof(float) + 255) / 256 * 256;
}

size_t sample_workspace_bytes(int n, int vocab) {
  const int nchunks = (vocab + kSampleChunk - 1) / kSampleChunk;
  return partial_bytes(n, nchunks) + 2 * list_bytes(n, nchunks);
}

bool sample_conf_supported(int vocab, int list_len) {
  const int nchunks = (vocab + kSampleChunk - 1) / kSampleChunk;
  return list_len >= 0 && list_len <= kConfMaxK && list_len <= vocab &&
         (size_t)nchunks * list_len <= (size_t)4 * kWave * kConfMergeNV;
}

hipError_t launch_logprob_sample(const float* logits, int n, int vocab, int64_t ld, float temp,
                                 uint64_t seed, const uint64_t* uid, const int32_t* positions,
                                 int32_t* out_tokens, float* out_lp, float* workspace,
                                 int conf_k, float* out_conf, float* conf_sum, hipStream_t st,
                                 int top_k, float top_p, float min_p) {
  if (n == 0) return hipSuccess;
  const int nchunks = (vocab + kSampleChunk - 1) / kSampleChunk;
  SamplePartial* part = reinterpret_cast<SamplePartial*>(workspace);
  char* lists = reinterpret_cast<char*>(workspace) + partial_bytes(n, nchunks);
  float* topk = reinterpret_cast<float*>(lists);
  int* topi = reinterpret_cast<int*>(lists + list_bytes(n, nchunks));
  if (top_k > 0) {
    const int L = top_k > conf_k ? top_k : conf_k;
    hipLaunchKernelGGL(sample_trunc_partial_kernel, dim3(nchunks, n), dim3(256), 0, st, logits,
                       vocab, ld, L, part, topk, topi);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(sample_trunc_final_kernel, dim3(n), dim3(256), 0, st, part, nchunks, L,
                       topk, topi, temp, top_k, top_p, min_p, seed, uid, positions, out_tokens,
                       out_lp, conf_k, out_conf, conf_sum);
    return hipGetLastError();
  }
  using PartialFn = void (*)(const float*, int, int64_t, float, uint64_t, const uint64_t*,
                            const int32_t*, SamplePartial*, int, float*);
  static constexpr PartialFn kPartial[3][2] = {
      {sample_partial_kernel<0, false>, sample_partial_kernel<0, true>},
      {sample_partial_kernel<1, false>, sample_partial_kernel<1, true>},
      {sample_partial_kernel<2, false>, sample_partial_kernel<2, true>}};
  const int mode = temp == 0.f ? 0 : temp == 1.f ? 1 : 2;
  hipLaunchKernelGGL(kPartial[mode][conf_k > 0 ? 1 : 0], dim3(nchunks, n), dim3(256), 0, st,
                     logits, vocab, ld, temp, seed, uid, positions, part, conf_k, topk);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sample_final_kernel, dim3(n), dim3(256), 0, st, part, nchunks, logits, vocab,
                     ld, temp, out_tokens, out_lp, conf_k, topk, out_conf, conf_sum);
  return hipGetLastError();
}

// One workgroup per sequence: binary search of its scored rows, then each
// thread sums a contiguous slice in order and the slices are added in thread
// order (a fixed order: the result does not depend on scheduling).
__global__ __launch_bounds__(256) void seq_confidence_kernel(const float* __restrict__ row_conf,
                                                             const int32_t* __restrict__ rows,
                                                             int n_scored,
                                                             const int32_t* __restrict__ seq_starts,
                                                             float* __restrict__ out) {
  __shared__ float part[256];
  const int s = blockIdx.x;
  auto lower = [&](int key) {  // first r with rows[r] >= key
    int lo = 0, hi = n_scored;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (rows[mid] < key) lo = mid + 1;
      else hi = mid;
    }
    return lo;
  };
  const int a = lower(seq_starts[s]), b = lower(seq_starts[s + 1]);
  const int n = b - a;
  const int per = (n + 255) / 256;
  const int r0 = a + threadIdx.x * per, r1 = min(b, r0 + per);
  float acc = 0.f;
  for (int r = r0; r < r1; ++r) acc += row_conf[r];
  part[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.f;
    for (int i = 0; i < 256; ++i) t += part[i];
    out[s] = n > 0 ? t / (float)n : 0.f;
  }
}

hipError_t launch_seq_confidence(const float* row_conf, const int32_t* scored_rows, int n_scored,
                                 const int32_t* seq_starts, int n_seqs, float* out,
                                 hipStream_t st) {
  if (n_seqs == 0) return hipSuccess;
  hipLaunchKernelGGL(seq_confidence_kernel, dim3(n_seqs), dim3(256), 0, st, row_conf, scored_rows,
                     n_scored, seq_starts, out);
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
