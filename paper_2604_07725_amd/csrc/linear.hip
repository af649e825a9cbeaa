// Skinny bf16 GEMM Y = X W^T on the gfx950 matrix cores, for the QKV, output,
// gate/up and down projections and the LM head of a decode step.
//
// At decode the batch M is the population size (<= 64 per tile), so the
// arithmetic intensity is M flop per weight byte: far below the MFMA ridge,
// the kernel is a weight stream and is designed for HBM bandwidth.
//   * one 256-thread workgroup per (64 output columns, K split, 64-row M tile)
//   * every wave covers all 64 columns x 16*MB rows with
//     v_mfma_f32_16x16x32_bf16 tiles and walks every fourth 32-wide k step of
//     the workgroup's K range, so the four waves of a workgroup read adjacent
//     64-byte pieces of the same weight rows;
//   * A operand = 16 weight rows x 32 k (one 16-byte load per lane),
//     B operand = 16 activation rows x 32 k (one 16-byte load per lane, L2
//     resident: the activations are tiny);
//   * the four waves' fp32 tiles are summed through LDS; split-K partials are
//     summed in split order by the epilogue kernel, which also applies the
//     residual add or the SwiGLU product.
#include "common.h"
#include "kernels.h"

namespace sevo {

template <int MB>
__global__ __launch_bounds__(256) void linear_kernel(const bf16_t* __restrict__ X, int ldx, int M,
                                                     const bf16_t* __restrict__ W, int N, int K,
                                                     int k_chunk, float* __restrict__ out,
                                                     int accumulate) {
  __shared__ f32x4 red[4][4][MB][64];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * 64;
  const int s = blockIdx.y;
  const int m0 = blockIdx.z * 16 * MB;
  const int r = lane & 15, q = lane >> 4;
  const int kb = s * k_chunk;
  const int ke = min(K, kb + k_chunk);

  const bf16_t* wp[4];
#pragma unroll
  for (int tt = 0; tt < 4; ++tt) wp[tt] = W + (size_t)(n0 + 16 * tt + r) * K + 8 * q;
  const bf16_t* xp[MB];
  bool xok[MB];
#pragma unroll
  for (int b = 0; b < MB; ++b) {
    const int row = m0 + 16 * b + r;
    xok[b] = row < M;
    xp[b] = X + (size_t)(xok[b] ? row : 0) * ldx + 8 * q;
  }

  f32x4 acc[4][MB];
#pragma unroll
  for (int tt = 0; tt < 4; ++tt)
#pragma unroll
    for (int b = 0; b < MB; ++b) acc[tt][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int k = kb + wave * 32; k < ke; k += 128) {
    bf16x8v a[4], bx[MB];
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
      a[tt] = __builtin_nontemporal_load(reinterpret_cast<const bf16x8v*>(wp[tt] + k));
#pragma unroll
    for (int b = 0; b < MB; ++b) {
      bf16x8v v = *reinterpret_cast<const bf16x8v*>(xp[b] + k);
      bx[b] = xok[b] ? v : bf16x8v{};
    }
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
      for (int b = 0; b < MB; ++b)
        acc[tt][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[tt], bx[b], acc[tt][b], 0, 0, 0);
  }

#pragma unroll
  for (int tt = 0; tt < 4; ++tt)
#pragma unroll
    for (int b = 0; b < MB; ++b) red[wave][tt][b][lane] = acc[tt][b];
  __syncthreads();
  // D[i][j] of tile (tt, b): lane holds j = lane % 16 (activation row) and
  // i = 4 (lane / 16) + 0..3 (weight row) -> 4 consecutive output columns.
  for (int idx = threadIdx.x; idx < 4 * MB * 64; idx += 256) {
    const int l = idx & 63;
    const int tb = idx >> 6;
    const int tt = tb / MB, b = tb - (tb / MB) * MB;
    const f32x4 v = red[0][tt][b][l] + red[1][tt][b][l] + red[2][tt][b][l] + red[3][tt][b][l];
    const int m = m0 + 16 * b + (l & 15);
    const int n = n0 + 16 * tt + 4 * (l >> 4);
    if (m < M) {
      f32x4* dst = reinterpret_cast<f32x4*>(out + (size_t)s * M * N + (size_t)m * N + n);
      if (accumulate) *dst = *dst + v;
      else *dst = v;
    }
  }
}

// Sum split-K partials in split order and apply the epilogue.
__global__ __launch_bounds__(256) void linear_epilogue_kernel(const float* __restrict__ part,
                                                              int S, int M, int N, int mode,
                                                              float* __restrict__ out_f32,
                                                              bf16_t* __restrict__ out_bf16) {
  const size_t MN = (size_t)M * N;
  const int F = N / 2;
  const size_t total4 = (mode == 2 ? (size_t)M * F : MN) / 4;
  for (size_t g = (size_t)blockIdx.x * blockDim.x + threadIdx.x; g < total4;
       g += (size_t)gridDim.x * blockDim.x) {
    if (mode == 2) {
      const size_t e = g * 4;
      const size_t m = e / F;
      const size_t j = e - m * F;
      f32x4 gs = f32x4{0.f, 0.f, 0.f, 0.f}, us = gs;
      for (int s = 0; s < S; ++s) {
        gs += *reinterpret_cast<const f32x4*>(part + s * MN + m * N + j);
        us += *reinterpret_cast<const f32x4*>(part + s * MN + m * N + F + j);
      }
      uint2 o;
      o.x = pack_bf16x2(gs.x / (1.f + expf(-gs.x)) * us.x, gs.y / (1.f + expf(-gs.y)) * us.y);
      o.y = pack_bf16x2(gs.z / (1.f + expf(-gs.z)) * us.z, gs.w / (1.f + expf(-gs.w)) * us.w);
      *reinterpret_cast<uint2*>(out_bf16 + m * F + j) = o;
    } else {
      f32x4 a = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int s = 0; s < S; ++s) a += *reinterpret_cast<const f32x4*>(part + s * MN + g * 4);
      f32x4* dst = reinterpret_cast<f32x4*>(out_f32 + g * 4);
      if (mode == 1) *dst = *dst + a;
      else *dst = a;
    }
  }
}

LinearPlan plan_linear(int m, int n_out, int k, int k_splits) {
  LinearPlan p;
  if (k_splits <= 0) {
    const int tiles = (n_out / 64) * ((m + 63) / 64);
    int s = 1;
    while (tiles * s < 512 && k / (2 * s) >= 512) s *= 2;
    k_splits = s;
  }
  int chunk = (k + k_splits - 1) / k_splits;
  chunk = (chunk + 127) / 128 * 128;
  p.k_chunk = chunk;
  p.k_splits = (k + chunk - 1) / chunk;
  return p;
}

size_t linear_workspace_bytes(int m, int n_out, int k, int k_splits) {
  // partials are needed when the K range is split or the epilogue is SwiGLU
  const LinearPlan p = plan_linear(m, n_out, k, k_splits);
  return (size_t)p.k_splits * m * n_out * sizeof(float);
}

hipError_t launch_linear(int m, int n_out, int k, int ldx, int mode, const LinearPlan& plan,
                         const bf16_t* x, const bf16_t* w, void* out, float* workspace,
                         hipStream_t st) {
  if (m == 0) return hipSuccess;
  const bool direct = plan.k_splits == 1 && mode != 2;
  float* dst = direct ? reinterpret_cast<float*>(out) : workspace;
  const int mtiles = (m + 63) / 64;
  const int mb = m >= 64 ? 4 : (m > 32 ? 4 : (m > 16 ? 2 : 1));
  dim3 grid(n_out / 64, plan.k_splits, m > 64 ? mtiles : 1);
  const int acc = direct && mode == 1 ? 1 : 0;
  if (m > 64 || mb == 4)
    hipLaunchKernelGGL(linear_kernel<4>, grid, dim3(256), 0, st, x, ldx, m, w, n_out, k,
                       plan.k_chunk, dst, acc);
  else if (mb == 2)
    hipLaunchKernelGGL(linear_kernel<2>, grid, dim3(256), 0, st, x, ldx, m, w, n_out, k,
                       plan.k_chunk, dst, acc);
  else
    hipLaunchKernelGGL(linear_kernel<1>, grid, dim3(256), 0, st, x, ldx, m, w, n_out, k,
                       plan.k_chunk, dst, acc);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || direct) return e;
  const size_t total4 = (mode == 2 ? (size_t)m * (n_out / 2) : (size_t)m * n_out) / 4;
  size_t blocks = (total4 + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(linear_epilogue_kernel, dim3((unsigned)blocks), dim3(256), 0, st, workspace,
                     plan.k_splits, m, n_out, mode, reinterpret_cast<float*>(out),
                     reinterpret_cast<bf16_t*>(out));
  return hipGetLastError();
}

}  // namespace sevo
