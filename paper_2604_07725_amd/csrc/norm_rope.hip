// Embedding gather, RMSNorm, fused QK-RMSNorm + RoPE + paged KV append, and
// the device twin of the synthetic-input generator.  All are tiny next to the
// attention and weight streams of a decode step; they are written for
// coalesced 16-byte accesses and one workgroup (or wave) per row / head.
#include "common.h"
#include "kernels.h"

namespace sevo {

// x[i][:] = embed[tokens[i]][:] (bf16 -> fp32).  One 256-thread block per row,
// 8 bf16 (16 B) per thread per step.  Out-of-range ids produce a zero row.
__global__ __launch_bounds__(256) void embed_kernel(const bf16_t* __restrict__ embed,
                                                    const int32_t* __restrict__ tokens,
                                                    int hidden, int vocab, float* __restrict__ x) {
  const int i = blockIdx.x;
  const int tok = tokens[i];
  const bool ok = tok >= 0 && tok < vocab;
  const bf16_t* src = embed + (size_t)(ok ? tok : 0) * hidden;
  float* dst = x + (size_t)i * hidden;
  for (int c = threadIdx.x * 8; c < hidden; c += 256 * 8) {
    u32x4 w = *reinterpret_cast<const u32x4*>(src + c);
    float4 a, b;
    a.x = ok ? bf16_lo(w.x) : 0.f; a.y = ok ? bf16_hi(w.x) : 0.f;
    a.z = ok ? bf16_lo(w.y) : 0.f; a.w = ok ? bf16_hi(w.y) : 0.f;
    b.x = ok ? bf16_lo(w.z) : 0.f; b.y = ok ? bf16_hi(w.z) : 0.f;
    b.z = ok ? bf16_lo(w.w) : 0.f; b.w = ok ? bf16_hi(w.w) : 0.f;
    *reinterpret_cast<float4*>(dst + c) = a;
    *reinterpret_cast<float4*>(dst + c + 4) = b;
  }
}

// out[r][:] = bf16(x[r][:] * (1 / sqrt(mean(x^2) + eps)) * gain).
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* __restrict__ x,
                                                      const bf16_t* __restrict__ gain, int cols,
                                                      float eps, bf16_t* __restrict__ out) {
  __shared__ float red[4];
  const float* xr = x + (size_t)blockIdx.x * cols;
  float ss = 0.f;
  for (int c = threadIdx.x * 4; c < cols; c += 1024) {
    float4 v = *reinterpret_cast<const float4*>(xr + c);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = block_sum<4>(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)cols + eps);
  bf16_t* orow = out + (size_t)blockIdx.x * cols;
  for (int c = threadIdx.x * 4; c < cols; c += 1024) {
    float4 v = *reinterpret_cast<const float4*>(xr + c);
    uint2 g = *reinterpret_cast<const uint2*>(gain + c);
    uint2 o;
    o.x = pack_bf16x2(v.x * inv * bf16_lo(g.x), v.y * inv * bf16_hi(g.x));
    o.y = pack_bf16x2(v.z * inv * bf16_lo(g.y), v.w * inv * bf16_hi(g.y));
    *reinterpret_cast<uint2*>(orow + c) = o;
  }
}

// One wave per (candidate, head) of the QKV projection (given as the fp32
// split-K partials of the GEMM, summed here in split order).  Lane m < d/2 owns
// the rotate-half pair (m, m + d/2).  q heads -> q_out; k heads -> K pool slot
// p_i; v heads -> V pool slot p_i (dim-major tile).  Positions outside the
// RoPE table or page ids outside the pool skip the write (no fault).
__global__ __launch_bounds__(64) void qk_norm_rope_append_kernel(RopeAppendArgs a) {
  const int i = blockIdx.x;
  const int hh = blockIdx.y;
  const int m = threadIdx.x;
  const int half = a.d >> 1;
  const bool act = m < half;
  const int qkv_ld = (a.hq + 2 * a.hkv) * a.d;
  const size_t split_stride = (size_t)a.n * qkv_ld;
  const float* src = a.qkv + (size_t)i * qkv_ld + (size_t)hh * a.d;
  float u0 = 0.f, u1 = 0.f;
  if (act) {
    for (int sp = 0; sp < a.qkv_splits; ++sp) {  // split-K partials, in split order
      u0 += src[sp * split_stride + m];
      u1 += src[sp * split_stride + m + half];
    }
  }
  const int p = a.positions[i];
  const bool pos_ok = p >= 0 && p < a.max_pos;
  const int prow = a.row_of_token ? a.row_of_token[i] : i;
  if (hh < a.hq + a.hkv) {
    if (a.qk_norm) {
      const float ss = wave_sum(u0 * u0 + u1 * u1);
      const float inv = 1.0f / sqrtf(ss / (float)a.d + a.eps);
      const bf16_t* g = hh < a.hq ? a.q_gain : a.k_gain;
      if (act) {
        u0 = u0 * inv * bf16_to_f32(g[m]);
        u1 = u1 * inv * bf16_to_f32(g[m + half]);
      }
    }
    if (!act) return;
    float r0 = 0.f, r1 = 0.f;
    if (pos_ok) {
      const float c = a.rope_cos[(size_t)p * half + m];
      const float s = a.rope_sin[(size_t)p * half + m];
      r0 = u0 * c - u1 * s;
      r1 = u1 * c + u0 * s;
    }
    if (hh < a.hq) {
      bf16_t* dst = a.q_out + ((size_t)i * a.hq + hh) * a.d;
      dst[m] = f32_to_bf16(r0);
      dst[m + half] = f32_to_bf16(r1);
      return;
    }
    if (!pos_ok) return;
    const int pg = p >> 4;
    if (pg >= a.max_pages) return;
    const int page = a.page_table[(size_t)prow * a.max_pages + pg];
    if (page < 0 || (int64_t)page >= a.num_pages) return;
    const int kh = hh - a.hq;
    // K tile (first half of the (page, head) pair): dims in blocks of 32, each
    // block [16 slots][32 dims]
    bf16_t* tile = a.kv_pool + ((size_t)page * a.hkv + kh) * 2 * kPage * a.d;
    const int s = p & 15;
    const int e0 = m, e1 = m + half;
    tile[((e0 >> 5) * kPage + s) * 32 + (e0 & 31)] = f32_to_bf16(r0);
    tile[((e1 >> 5) * kPage + s) * 32 + (e1 & 31)] = f32_to_bf16(r1);
  } else {
    if (!act || !pos_ok) return;
    const int pg = p >> 4;
    if (pg >= a.max_pages) return;
    const int page = a.page_table[(size_t)prow * a.max_pages + pg];
    if (page < 0 || (int64_t)page >= a.num_pages) return;
    const int vh = hh - a.hq - a.hkv;
    // V tile (second half): dim-major [dims][16 slots]
    bf16_t* dst = a.kv_pool + (((size_t)page * a.hkv + vh) * 2 + 1) * kPage * a.d + (p & 15);
    dst[(size_t)m * kPage] = f32_to_bf16(u0);
    dst[(size_t)(m + half) * kPage] = f32_to_bf16(u1);
  }
}

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ bf16_t synth_value(uint64_t key, int64_t e, float mul, float add,
                                              int use_add) {
  const uint64_t r = mix64(key + (uint64_t)(e + 1) * 0x9E3779B97F4A7C15ull);
  const int32_t s = (int32_t)(r & 0xFFFF) + (int32_t)((r >> 16) & 0xFFFF) +
                    (int32_t)((r >> 32) & 0xFFFF) + (int32_t)(r >> 48);
  float v = __fmul_rn((float)(s - 131070), mul);
  if (use_add) v = __fadd_rn(v, add);
  return f32_to_bf16(v);
}

// Eight elements (one 16-byte store) per thread per step; scalar tail.
__global__ __launch_bounds__(256) void fill_bf16_kernel(bf16_t* __restrict__ dst, int64_t count,
                                                        uint64_t key, int64_t offset, float mul,
                                                        float add, int use_add) {
  const int64_t n8 = count >> 3;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < n8; g += stride) {
    const int64_t e = g << 3;
    u32x4 w;
    w.x = synth_value(key, offset + e, mul, add, use_add) |
          ((uint32_t)synth_value(key, offset + e + 1, mul, add, use_add) << 16);
    w.y = synth_value(key, offset + e + 2, mul, add, use_add) |
          ((uint32_t)synth_value(key, offset + e + 3, mul, add, use_add) << 16);
    w.z = synth_value(key, offset + e + 4, mul, add, use_add) |
          ((uint32_t)synth_value(key, offset + e + 5, mul, add, use_add) << 16);
    w.w = synth_value(key, offset + e + 6, mul, add, use_add) |
          ((uint32_t)synth_value(key, offset + e + 7, mul, add, use_add) << 16);
    *reinterpret_cast<u32x4*>(dst + e) = w;
  }
  const int64_t tail0 = n8 << 3;
  const int64_t t = tail0 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < count && t - tail0 < 8) dst[t] = synth_value(key, offset + t, mul, add, use_add);
}

hipError_t launch_embed(const bf16_t* embed, const int32_t* tokens, int n, int hidden, int vocab,
                        float* x, hipStream_t st) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(embed_kernel, dim3(n), dim3(256), 0, st, embed, tokens, hidden, vocab, x);
  return hipGetLastError();
}

// x[r] += sum_s part[s][r] in split order, written back; then the RMSNorm,
// stored in the tiled activation layout that the projections read.
// 1024 threads per row, each owning 4 consecutive columns per 4096-column
// pass with all split loads independent (latency, not bandwidth, is the cost).
// With row_idx, output row r reads row row_idx[r] of x and the partials and
// x is not written back (the final norm of a prefill's scored rows).
__global__ __launch_bounds__(1024) void add_rmsnorm_kernel(float* __restrict__ x,
                                                           const float* __restrict__ part, int S,
                                                           size_t part_stride,
                                                           const bf16_t* __restrict__ gain,
                                                           int cols, float eps,
                                                           bf16_t* __restrict__ out,
                                                           const int32_t* __restrict__ row_idx) {
  __shared__ float red[16];
  const size_t src = row_idx ? (size_t)row_idx[blockIdx.x] : (size_t)blockIdx.x;
  float* xr = x + src * cols;
  const float* pr = part + src * cols;
  float ss = 0.f;
  for (int c = threadIdx.x * 4; c < cols; c += 4096) {
    f32x4 v = *reinterpret_cast<const f32x4*>(xr + c);
    if (S > 0) {
      f32x4 p[16];
#pragma unroll
      for (int s = 0; s < 16; ++s)
        if (s < S) p[s] = *reinterpret_cast<const f32x4*>(pr + s * part_stride + c);
#pragma unroll
      for (int s = 0; s < 16; ++s)
        if (s < S) v += p[s];
      if (!row_idx) *reinterpret_cast<f32x4*>(xr + c) = v;
    }
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = block_sum<16>(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)cols + eps);
  for (int c = threadIdx.x * 4; c < cols; c += 4096) {
    f32x4 v = *reinterpret_cast<const f32x4*>(xr + c);
    if (row_idx) {  // x was not updated in place: add the partials again, same order
      f32x4 p[16];
#pragma unroll
      for (int s = 0; s < 16; ++s)
        if (s < S) p[s] = *reinterpret_cast<const f32x4*>(pr + s * part_stride + c);
#pragma unroll
      for (int s = 0; s < 16; ++s)
        if (s < S) v += p[s];
    }
    const uint2 g = *reinterpret_cast<const uint2*>(gain + c);
    uint2 o;
    o.x = pack_bf16x2(v.x * inv * bf16_lo(g.x), v.y * inv * bf16_hi(g.x));
    o.y = pack_bf16x2(v.z * inv * bf16_lo(g.y), v.w * inv * bf16_hi(g.y));
    // 4 consecutive columns are contiguous in the tiled activation layout
    *reinterpret_cast<uint2*>(out + act_tile_offset(blockIdx.x, c, cols)) = o;
  }
}

hipError_t launch_add_rmsnorm(float* x, const float* part, int S, const bf16_t* gain, int rows,
                              int cols, float eps, bf16_t* out_tiled, hipStream_t st,
                              const int32_t* row_idx, int part_rows) {
  if (rows == 0) return hipSuccess;
  if (S > 16) return hipErrorInvalidValue;
  const size_t stride = (size_t)(row_idx ? part_rows : rows) * cols;
  hipLaunchKernelGGL(add_rmsnorm_kernel, dim3(rows), dim3(1024), 0, st, x, part, part ? S : 0,
                     stride, gain, cols, eps, out_tiled, row_idx);
  return hipGetLastError();
}

// Packed token t of a prefill batch -> its sequence s (the page-table row)
// and position start_pos[s] + t - seq_starts[s].
__global__ __launch_bounds__(256) void prefill_index_kernel(const int32_t* __restrict__ seq_starts,
                                                            const int32_t* __restrict__ start_pos,
                                                            int n_seqs, int T,
                                                            int32_t* __restrict__ row,
                                                            int32_t* __restrict__ pos) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= T) return;
  int lo = 0, hi = n_seqs - 1;  // last s with seq_starts[s] <= t
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (seq_starts[mid] <= t) lo = mid;
    else hi = mid - 1;
  }
  row[t] = lo;
  pos[t] = (start_pos ? start_pos[lo] : 0) + t - seq_starts[lo];
}

hipError_t launch_prefill_index(const int32_t* seq_starts, const int32_t* start_pos, int n_seqs,
                                int T, int32_t* row, int32_t* pos, hipStream_t st) {
  if (T == 0) return hipSuccess;
  hipLaunchKernelGGL(prefill_index_kernel, dim3((T + 255) / 256), dim3(256), 0, st, seq_starts,
                     start_pos, n_seqs, T, row, pos);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(const float* x, const bf16_t* gain, int rows, int cols, float eps,
                          bf16_t* out, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(rmsnorm_kernel, dim3(rows), dim3(256), 0, st, x, gain, cols, eps, out);
  return hipGetLastError();
}

hipError_t launch_qk_norm_rope_append(const RopeAppendArgs& a, hipStream_t st) {
  if (a.n == 0) return hipSuccess;
  hipLaunchKernelGGL(qk_norm_rope_append_kernel, dim3(a.n, a.hq + 2 * a.hkv), dim3(64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_fill_bf16(bf16_t* dst, int64_t count, uint64_t key, int64_t offset, float mul,
                            float add, int use_add, hipStream_t st) {
  if (count == 0) return hipSuccess;
  int64_t blocks = ((count >> 3) + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(fill_bf16_kernel, dim3((unsigned)blocks), dim3(256), 0, st, dst, count, key,
                     offset, mul, add, use_add);
  return hipGetLastError();
}

}  // namespace sevo
