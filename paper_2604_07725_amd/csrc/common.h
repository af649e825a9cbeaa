// Device-side helpers shared by the gfx950 kernels of libsevo.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sevo {

typedef uint16_t bf16_t;
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8v __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kPage = 16;

// ---- GEMM operand layouts (bf16), built around one MFMA 16x16x32 fragment:
// 16 rows x 32 columns stored as 64 lanes x 8 values, lane = 16 (c/8 % 4) + r % 16,
// so a wave loads a whole fragment as one contiguous 1 KB read.
//
// Packed weight [n_out][k]: superblocks of 64 rows; for each 32-column step
// the superblock's four 16-row fragments are adjacent (2048 elements), so a
// workgroup streaming a superblock reads one contiguous region.
__host__ __device__ __forceinline__ size_t packed_weight_offset(int r, int c, int k) {
  return (((size_t)(r >> 6) * (k >> 5) + (c >> 5)) * 4 + ((r >> 4) & 3)) * 512 +
         (((c >> 3) & 3) * 16 + (r & 15)) * 8 + (c & 7);
}
// Tiled activation [m][k]: 16-row blocks, each a run of k/32 fragments.
// Rows are padded to a multiple of 16 (padding rows are never read into a
// stored output).
__host__ __device__ __forceinline__ size_t act_tile_offset(int m, int c, int k) {
  return ((size_t)(m >> 4) * (k >> 5) + (c >> 5)) * 512 + (((c >> 3) & 3) * 16 + (m & 15)) * 8 +
         (c & 7);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ float bf16_to_f32(bf16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round-to-nearest-even fp32 -> bf16: gfx950 converts in hardware
// (v_cvt_pk_bf16_f32, two values per instruction).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(bf16_t, (__bf16)f);
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2v v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// a.x*b.x + a.y*b.y + c, bf16 pairs packed in 32-bit words, fp32 accumulate.
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2v, a),
                                         __builtin_bit_cast(bf16x2v, b), c, false);
}

// ---- cross-lane reductions in registers (DPP and the gfx950 permlane swaps;
// no LDS round trip).  Lane groups follow the wave64 layout: quads of 4
// lanes, rows of 16 lanes, halves of 32 lanes.
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppQuadXor1 = 0xB1;  // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;  // quad_perm [2,3,0,1]
constexpr int kDppRowRor4 = 0x124;
constexpr int kDppRowRor8 = 0x128;
constexpr int kDppRowMirror = 0x140;      // lane i <- lane 15 - i of its row
constexpr int kDppRowHalfMirror = 0x141;  // lane i <- lane 7 - i of its 8-lane half row

// sum over the 4 lanes of each quad (every lane gets the result)
__device__ __forceinline__ float quad_sum(float v) {
  v += dpp<kDppQuadXor1>(v);
  return v + dpp<kDppQuadXor2>(v);
}
// combine lane i with lane i ^ 16 (rows 0<->1, 2<->3), every lane gets the result
__device__ __forceinline__ float xor16_max(float v) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_int(v), __float_as_int(v), false, false);
  return fmaxf(__int_as_float(p[0]), __int_as_float(p[1]));
}
__device__ __forceinline__ float xor16_sum(float v) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_int(v), __float_as_int(v), false, false);
  return __int_as_float(p[0]) + __int_as_float(p[1]);
}
// combine lane i with lane i ^ 32
__device__ __forceinline__ float xor32_max(float v) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_int(v), __float_as_int(v), false, false);
  return fmaxf(__int_as_float(p[0]), __int_as_float(p[1]));
}
__device__ __forceinline__ float xor32_sum(float v) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_int(v), __float_as_int(v), false, false);
  return __int_as_float(p[0]) + __int_as_float(p[1]);
}
// max / sum over the lanes with equal lane % 4 (the quads of the wave)
__device__ __forceinline__ float quads_max(float v) {
  v = fmaxf(v, dpp<kDppRowRor4>(v));
  v = fmaxf(v, dpp<kDppRowRor8>(v));
  return xor32_max(xor16_max(v));
}
__device__ __forceinline__ float quads_sum(float v) {
  v += dpp<kDppRowRor4>(v);
  v += dpp<kDppRowRor8>(v);
  return xor32_sum(xor16_sum(v));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// Block-wide sum for blockDim.x == 64 * NW; every thread gets the result.
template <int NW>
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < NW; ++i) t += red[i];
  __syncthreads();
  return t;
}

// ---- wait counters and a fence-free barrier, for kernels that stream
// through LDS with direct global -> LDS loads.
// Waits until at most N vector-memory operations of this wave are
// outstanding (gfx9 s_waitcnt: vmcnt split over bits 3:0 and 15:14, expcnt
// and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
// Waits for all LDS reads of this wave (lgkmcnt 0, the others at maxima).
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xC07F); }
// Workgroup barrier without the release/acquire fences of __syncthreads:
// those make the compiler wait for every outstanding direct load (vmcnt 0),
// which would drain a multi-stage pipeline.  Each wave waits for exactly the
// loads the next stage needs (wait_vmcnt) and for its own LDS reads
// (wait_lgkm0) before arriving; the memory clobber keeps the compiler from
// moving LDS accesses across the barrier.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}
// Direct global -> LDS load of 16 bytes per lane through a buffer descriptor:
// lane i's bytes land at lds_wave_base + 16 i.  The descriptor's record count
// bounds every access (offsets past it read zeros and touch no memory).
template <typename T>
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, uint32_t voff, T* lds_wave_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(
      r, (__attribute__((address_space(3))) void*)lds_wave_base, 16, (int)voff, 0, 0, 0);
}

}  // namespace sevo
