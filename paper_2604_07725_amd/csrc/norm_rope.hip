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

// What lane m needs of token i for every head: position, its K/V page (-1:
// no append), the RoPE cos / sin of the pair (m, m + d/2) and the QK-norm
// gains.  Positions outside the RoPE table or page ids outside the pool skip
// the writes (no fault).
struct RopeTok {
  int p, page;
  bool pos_ok;
  float c, s, gq0, gq1, gk0, gk1;
};

__device__ __forceinline__ RopeTok rope_token(const RopeAppendArgs& a, int i, int m) {
  const int half = a.d >> 1;
  RopeTok t{};
  t.p = a.positions[i];
  t.pos_ok = t.p >= 0 && t.p < a.max_pos;
  t.page = -1;
  if (m < half) {
    if (t.pos_ok) {
      t.c = a.rope_cos[(size_t)t.p * half + m];
      t.s = a.rope_sin[(size_t)t.p * half + m];
      const int pg = t.p >> 4;
      if (pg < a.max_pages) {
        const int prow = a.row_of_token ? a.row_of_token[i] : i;
        const int page = a.page_table[(size_t)prow * a.max_pages + pg];
        if (page >= 0 && (int64_t)page < a.num_pages) t.page = page;
      }
    }
    if (a.qk_norm) {
      t.gq0 = bf16_to_f32(a.q_gain[m]);
      t.gq1 = bf16_to_f32(a.q_gain[m + half]);
      t.gk0 = bf16_to_f32(a.k_gain[m]);
      t.gk1 = bf16_to_f32(a.k_gain[m + half]);
    }
  }
  return t;
}

// QK-RMSNorm + RoPE + store of one (token i, head hh) of the QKV projection,
// called by a whole wave with the summed values u0 = row[m], u1 = row[m + d/2]
// in lane m < d/2 (lane m owns the rotate-half pair).  q heads -> q_out; k
// heads -> K pool slot p_i; v heads -> V pool slot p_i (dim-major tile).
__device__ __forceinline__ void rope_head(const RopeAppendArgs& a, const RopeTok& t, int i,
                                          int hh, int m, float u0, float u1) {
  const int half = a.d >> 1;
  const bool act = m < half;
  if (hh < a.hq + a.hkv) {
    if (a.qk_norm) {
      const float ss = wave_sum(u0 * u0 + u1 * u1);
      const float inv = 1.0f / sqrtf(ss / (float)a.d + a.eps);
      const bool q = hh < a.hq;
      if (act) {
        u0 = u0 * inv * (q ? t.gq0 : t.gk0);
        u1 = u1 * inv * (q ? t.gq1 : t.gk1);
      }
    }
    if (!act) return;
    float r0 = 0.f, r1 = 0.f;
    if (t.pos_ok) {
      r0 = u0 * t.c - u1 * t.s;
      r1 = u1 * t.c + u0 * t.s;
    }
    if (hh < a.hq) {
      bf16_t* dst = a.q_out + ((size_t)i * a.hq + hh) * a.d;
      dst[m] = f32_to_bf16(r0);
      dst[m + half] = f32_to_bf16(r1);
      return;
    }
    if (t.page < 0) return;
    const int kh = hh - a.hq;
    // K tile (first half of the (page, head) pair): dims in blocks of 32, each
    // block [16 slots][32 dims]
    bf16_t* tile = a.kv_pool + ((size_t)t.page * a.hkv + kh) * 2 * kPage * a.d;
    const int s = t.p & 15;
    const int e0 = m, e1 = m + half;
    tile[((e0 >> 5) * kPage + s) * 32 + (e0 & 31)] = f32_to_bf16(r0);
    tile[((e1 >> 5) * kPage + s) * 32 + (e1 & 31)] = f32_to_bf16(r1);
  } else {
    if (!act || t.page < 0) return;
    const int vh = hh - a.hq - a.hkv;
    // V tile (second half): dim-major [dims][16 slots]
    bf16_t* dst = a.kv_pool + (((size_t)t.page * a.hkv + vh) * 2 + 1) * kPage * a.d + (t.p & 15);
    dst[(size_t)m * kPage] = f32_to_bf16(u0);
    dst[(size_t)(m + half) * kPage] = f32_to_bf16(u1);
  }
}

// Separate K and V pools [page][head][16 slots][d] (row-major slots) -> the
// fused pool [page][head][K tile | V tile] that the attention kernels read:
// one workgroup (2 d threads) per (page, head) pair, grid-stride.  Every
// thread moves 8 consecutive dims of one slot: K straight into its 32-dim
// block (a 16-byte store), V through LDS so that the dim-major V tile is
// written in 16-byte runs of 8 slots.
__global__ __launch_bounds__(256) void pack_kv_kernel(const bf16_t* __restrict__ k_src,
                                                      const bf16_t* __restrict__ v_src,
                                                      size_t tiles, int d,
                                                      bf16_t* __restrict__ kv) {
  __shared__ __align__(16) bf16_t vt[kPage * 128];
  const int t = threadIdx.x;
  const int s = t / (d >> 3), e0 = (t % (d >> 3)) * 8;  // slot, first dim
  const int e = t >> 1, h = t & 1;                      // V: dim, slot half
  const size_t tile_elems = (size_t)kPage * d;
  for (size_t tl = blockIdx.x; tl < tiles; tl += gridDim.x) {
    const size_t src = tl * tile_elems + (size_t)s * d + e0;
    const u32x4 kw = *reinterpret_cast<const u32x4*>(k_src + src);
    const u32x4 vw = *reinterpret_cast<const u32x4*>(v_src + src);
    bf16_t* kt = kv + tl * 2 * tile_elems;
    *reinterpret_cast<u32x4*>(kt + ((e0 >> 5) * kPage + s) * 32 + (e0 & 31)) = kw;
    __syncthreads();  // the previous tile's V reads are done
    *reinterpret_cast<u32x4*>(vt + s * d + e0) = vw;
    __syncthreads();
    uint16_t r[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) r[j] = __builtin_bit_cast(uint16_t, vt[(8 * h + j) * d + e]);
    u32x4 o;
    o.x = r[0] | ((uint32_t)r[1] << 16);
    o.y = r[2] | ((uint32_t)r[3] << 16);
    o.z = r[4] | ((uint32_t)r[5] << 16);
    o.w = r[6] | ((uint32_t)r[7] << 16);
    *reinterpret_cast<u32x4*>(kt + tile_elems + e * kPage + 8 * h) = o;
  }
}

hipError_t launch_pack_kv(const bf16_t* k_src, const bf16_t* v_src, size_t tiles, int d,
                          bf16_t* kv, hipStream_t st) {
  if (tiles == 0) return hipSuccess;
  const unsigned grid = (unsigned)(tiles < 65536 ? tiles : 65536);
  hipLaunchKernelGGL(pack_kv_kernel, dim3(grid), dim3(2 * d), 0, st, k_src, v_src, tiles, d, kv);
  return hipGetLastError();
}

// One wave per (candidate, head); the QKV projection given as the fp32
// split-K partials of the GEMM, summed here in split order.
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
    // split-K partials in split order; four splits' loads issued together
    // (a load per iteration would wait out one memory latency per split)
    for (int s0 = 0; s0 < a.qkv_splits; s0 += 4) {
      float v0[4], v1[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (s0 + j < a.qkv_splits) {
          v0[j] = src[(s0 + j) * split_stride + m];
          v1[j] = src[(s0 + j) * split_stride + m + half];
        }
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (s0 + j < a.qkv_splits) {
          u0 += v0[j];
          u1 += v1[j];
        }
    }
  }
  rope_head(a, rope_token(a, i, m), i, hh, m, u0, u1);
}

// The same per token, for many tokens (a prefill): one 4-wave workgroup per
// token, wave w taking heads w, w + 4, ...; the token's position, page, RoPE
// row and gains are loaded once and every head's values before any
// arithmetic (one wave per (token, head) left the launch of millions of
// one-wave workgroups as the cost).  Identical output.
constexpr int kRopeHeadsPerWave = 20;  // hq + 2 hkv <= 80
__global__ __launch_bounds__(256) void qk_norm_rope_append_token_kernel(RopeAppendArgs a) {
  const int i = blockIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), m = threadIdx.x & 63;
  const int half = a.d >> 1;
  const bool act = m < half;
  const int H = a.hq + 2 * a.hkv;
  const int qkv_ld = H * a.d;
  const size_t split_stride = (size_t)a.n * qkv_ld;
  const RopeTok t = rope_token(a, i, m);
  float u0[kRopeHeadsPerWave], u1[kRopeHeadsPerWave];
#pragma unroll
  for (int j = 0; j < kRopeHeadsPerWave; ++j) u0[j] = u1[j] = 0.f;
  for (int sp = 0; sp < a.qkv_splits; ++sp) {  // split-K partials, in split order
    // one descriptor over the token's row: the head offset is a scalar
    // offset, the lane's 4 m bytes the only per-lane address
    const __amdgpu_buffer_rsrc_t row = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(a.qkv + sp * split_stride + (size_t)i * qkv_ld), 0, qkv_ld * 4,
        0x00020000);
#pragma unroll
    for (int j = 0; j < kRopeHeadsPerWave; ++j) {
      const int hh = 4 * j + w;
      if (act && hh < H) {
        u0[j] += __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(row, m * 4, hh * a.d * 4, 0));
        u1[j] += __uint_as_float(
            __builtin_amdgcn_raw_buffer_load_b32(row, (m + half) * 4, hh * a.d * 4, 0));
      }
    }
  }
#pragma unroll
  for (int j = 0; j < kRopeHeadsPerWave; ++j) {
    const int hh = 4 * j + w;
    if (hh < H) rope_head(a, t, i, hh, m, u0[j], u1[j]);
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
  // x plus the partials (split order) at column c, written back to x
  auto load_sum = [&](int c) {
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
    return v;
  };
  auto store_out = [&](int c, f32x4 v, float inv) {
    const uint2 g = *reinterpret_cast<const uint2*>(gain + c);
    uint2 o;
    o.x = pack_bf16x2(v.x * inv * bf16_lo(g.x), v.y * inv * bf16_hi(g.x));
    o.y = pack_bf16x2(v.z * inv * bf16_lo(g.y), v.w * inv * bf16_hi(g.y));
    // 4 consecutive columns are contiguous in the tiled activation layout
    *reinterpret_cast<uint2*>(out + act_tile_offset(blockIdx.x, c, cols)) = o;
  };
  // the first two 4-column groups of a thread (every row up to 8192 columns)
  // stay in registers across the reduction instead of being read back from x
  const int c0 = threadIdx.x * 4, c1 = c0 + 4096;
  f32x4 v0 = f32x4{0.f, 0.f, 0.f, 0.f}, v1 = v0;
  float ss = 0.f;
  if (c0 < cols) {
    v0 = load_sum(c0);
    ss += v0.x * v0.x + v0.y * v0.y + v0.z * v0.z + v0.w * v0.w;
  }
  if (c1 < cols) {
    v1 = load_sum(c1);
    ss += v1.x * v1.x + v1.y * v1.y + v1.z * v1.z + v1.w * v1.w;
  }
  for (int c = c0 + 8192; c < cols; c += 4096) {
    const f32x4 v = load_sum(c);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = block_sum<16>(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)cols + eps);
  if (c0 < cols) store_out(c0, v0, inv);
  if (c1 < cols) store_out(c1, v1, inv);
  for (int c = c0 + 8192; c < cols; c += 4096) {
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
    store_out(c, v, inv);
  }
}

// The same for many rows with at most one partial (a prefill): 256 threads
// per row, so eight rows per CU are in flight instead of two, and thread t
// keeps the 4-column groups 1024 g + 4 t (g < NG) in registers across the
// reduction.  The sum of squares is formed exactly as in the 1024-thread form:
// the groups of its thread T = 256 (g % 4) + t in order, one wave sum per
// wave of T, the 16 wave sums in order, so both forms give identical output.
template <int NG>
__global__ __launch_bounds__(256) void add_rmsnorm_rows_kernel(float* __restrict__ x,
                                                               const float* __restrict__ part,
                                                               int S, const bf16_t* __restrict__ gain,
                                                               int cols, float eps,
                                                               bf16_t* __restrict__ out,
                                                               const int32_t* __restrict__ row_idx) {
  __shared__ float red[16];
  const size_t src = row_idx ? (size_t)row_idx[blockIdx.x] : (size_t)blockIdx.x;
  float* xr = x + src * cols;
  const float* pr = part + src * cols;
  const int t = threadIdx.x;
  f32x4 v[NG];
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int c = 1024 * g + 4 * t;
    if (c < cols) v[g] = *reinterpret_cast<const f32x4*>(xr + c);
  }
  if (S > 0) {
    f32x4 p[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const int c = 1024 * g + 4 * t;
      if (c < cols) p[g] = *reinterpret_cast<const f32x4*>(pr + c);
    }
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const int c = 1024 * g + 4 * t;
      if (c < cols) {
        v[g] += p[g];
        if (!row_idx) *reinterpret_cast<f32x4*>(xr + c) = v[g];
      }
    }
  }
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int c = 1024 * g + 4 * t;
    if (c < cols) acc[g & 3] += v[g].x * v[g].x + v[g].y * v[g].y + v[g].z * v[g].z + v[g].w * v[g].w;
  }
  const int w = t >> 6;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float sq = wave_sum(acc[q]);
    if ((t & 63) == 0) red[4 * q + w] = sq;
  }
  __syncthreads();
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < 16; ++i) ss += red[i];
  const float inv = 1.0f / sqrtf(ss / (float)cols + eps);
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int c = 1024 * g + 4 * t;
    if (c < cols) {
      const uint2 gn = *reinterpret_cast<const uint2*>(gain + c);
      uint2 o;
      o.x = pack_bf16x2(v[g].x * inv * bf16_lo(gn.x), v[g].y * inv * bf16_hi(gn.x));
      o.y = pack_bf16x2(v[g].z * inv * bf16_lo(gn.y), v[g].w * inv * bf16_hi(gn.y));
      *reinterpret_cast<uint2*>(out + act_tile_offset(blockIdx.x, c, cols)) = o;
    }
  }
}

hipError_t launch_add_rmsnorm(float* x, const float* part, int S, const bf16_t* gain, int rows,
                              int cols, float eps, bf16_t* out_tiled, hipStream_t st,
                              const int32_t* row_idx, int part_rows) {
  if (rows == 0) return hipSuccess;
  if (S > 16) return hipErrorInvalidValue;
  const size_t stride = (size_t)(row_idx ? part_rows : rows) * cols;
  const int s_eff = part ? S : 0;
  if (rows >= 512 && s_eff <= 1 && cols <= 8192) {
    const int ng = (cols + 1023) / 1024;
    auto go = [&](auto kern) {
      hipLaunchKernelGGL(kern, dim3(rows), dim3(256), 0, st, x, part, s_eff, gain, cols, eps,
                         out_tiled, row_idx);
    };
    if (ng <= 2) go(add_rmsnorm_rows_kernel<2>);
    else if (ng <= 4) go(add_rmsnorm_rows_kernel<4>);
    else go(add_rmsnorm_rows_kernel<8>);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(add_rmsnorm_kernel, dim3(rows), dim3(1024), 0, st, x, part, s_eff, stride,
                     gain, cols, eps, out_tiled, row_idx);
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
  if (a.n >= 256 && a.hq + 2 * a.hkv <= 4 * kRopeHeadsPerWave)
    hipLaunchKernelGGL(qk_norm_rope_append_token_kernel, dim3(a.n), dim3(256), 0, st, a);
  else
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
