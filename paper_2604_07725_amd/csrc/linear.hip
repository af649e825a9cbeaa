// Skinny bf16 GEMM Y = X W^T on the gfx950 matrix cores, for the QKV, output,
// gate/up and down projections and the LM head of a decode step.
//
// At decode the batch M is the population size (<= 64 per tile), so the
// arithmetic intensity is M flop per weight byte: far below the MFMA ridge,
// the kernel is a weight stream and is designed for HBM bandwidth.
//   * one 256-thread workgroup per (64 weight rows, K split, 64-row M tile);
//   * the four waves split the workgroup's K range into contiguous parts and
//     step 32 k at a time (one v_mfma_f32_16x16x32_bf16 k-block), so two
//     consecutive steps of one wave read whole 128-byte lines of its rows;
//   * A operand = 16 weight rows x 32 k (lane: row lane%16, k 8*(lane/16)..+7),
//     B operand = 16 activation rows x 32 k (L2 resident: activations are tiny);
//   * four register fragment buffers keep the next three steps' loads in
//     flight while the current step's MFMAs run;
//   * the four waves' fp32 tiles are summed through LDS.  With K split across
//     workgroups the fp32 partials [split][m][n] are summed, in split order, by
//     the consumer (the epilogue kernel here, or the fused norm / RoPE kernels
//     of the decode step).  The SwiGLU form pairs 32 gate rows with the
//     matching 32 up rows in one workgroup and writes silu(g) * u directly.
#include "common.h"
#include "kernels.h"

namespace sevo {

template <int MB>
struct GemmFrag {
  bf16x8v a[4];
  bf16x8v b[MB];
};

// EPI 0: fp32 tile (split partial, or final with optional accumulate)
// EPI 2: SwiGLU, bf16 out[m][F] (needs the full K range in one workgroup)
template <int MB, int EPI>
__global__ __launch_bounds__(256, 2) void linear_kernel(const bf16_t* __restrict__ X, int ldx,
                                                        int M, const bf16_t* __restrict__ W, int N,
                                                        int K, int k_chunk, float* __restrict__ out,
                                                        int accumulate,
                                                        bf16_t* __restrict__ out_bf16) {
  __shared__ f32x4 red[4][4][MB][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int s = blockIdx.y;
  const int m0 = blockIdx.z * 16 * MB;
  const int r = lane & 15, q = lane >> 4;
  const int F = N / 2;
  const int j0 = blockIdx.x * 32;  // SwiGLU: first gate column of this tile

  const bf16_t* wp[4];
#pragma unroll
  for (int tt = 0; tt < 4; ++tt) {
    int row;
    if constexpr (EPI == 2) row = (tt < 2 ? j0 : F + j0) + 16 * (tt & 1) + r;
    else row = blockIdx.x * 64 + 16 * tt + r;
    wp[tt] = W + (size_t)row * K + 8 * q;
  }
  // activation rows past M read row M-1: they only feed output rows that are
  // never stored, so no masking (and no wait on the loaded value) is needed
  const bf16_t* xp[MB];
#pragma unroll
  for (int b = 0; b < MB; ++b) {
    const int row = min(m0 + 16 * b + r, M - 1);
    xp[b] = X + (size_t)row * ldx + 8 * q;
  }

  // this wave's contiguous share of the workgroup's K range, in 32-k steps
  // (each pair of steps reads whole 128-byte lines of its weight rows)
  const int kb = s * k_chunk;
  const int ke = min(K, kb + k_chunk);
  const int nsteps = (ke - kb) >> 5;            // a multiple of 4 (k_chunk % 128 == 0)
  const int per = ((nsteps + 15) >> 4) << 2;   // steps per wave, a multiple of 4
  const int st0 = wave * per;
  const int st1 = min(nsteps, st0 + per);

  f32x4 acc[4][MB];
#pragma unroll
  for (int tt = 0; tt < 4; ++tt)
#pragma unroll
    for (int b = 0; b < MB; ++b) acc[tt][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto load = [&](GemmFrag<MB>& f, int st) {
    const int k = kb + st * 32;
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) f.a[tt] = *reinterpret_cast<const bf16x8v*>(wp[tt] + k);
#pragma unroll
    for (int b = 0; b < MB; ++b) f.b[b] = *reinterpret_cast<const bf16x8v*>(xp[b] + k);
  };
  auto mma = [&](const GemmFrag<MB>& f) {
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
      for (int b = 0; b < MB; ++b)
        acc[tt][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.a[tt], f.b[b], acc[tt][b], 0, 0, 0);
  };

  // Every wave owns a multiple of 4 steps, so the loop takes four per trip
  // with one exit, rotating four fragment buffers: while one is multiplied the
  // next three are in flight.  Prefetches past the end re-read the last step
  // (L2 hits).  sched_barrier keeps the scheduler from sinking the prefetch
  // loads next to their MFMAs, which would serialise the stream.
  if (st0 < st1) {
    GemmFrag<MB> f0, f1, f2, f3;
    load(f0, st0);
    load(f1, st0 + 1);
    load(f2, st0 + 2);
    for (int st = st0; st < st1; st += 4) {
      load(f3, st + 3);
      __builtin_amdgcn_sched_barrier(0);
      mma(f0);
      __builtin_amdgcn_sched_barrier(0);
      load(f0, min(st + 4, st1 - 1));
      __builtin_amdgcn_sched_barrier(0);
      mma(f1);
      __builtin_amdgcn_sched_barrier(0);
      load(f1, min(st + 5, st1 - 1));
      __builtin_amdgcn_sched_barrier(0);
      mma(f2);
      __builtin_amdgcn_sched_barrier(0);
      load(f2, min(st + 6, st1 - 1));
      __builtin_amdgcn_sched_barrier(0);
      mma(f3);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

#pragma unroll
  for (int tt = 0; tt < 4; ++tt)
#pragma unroll
    for (int b = 0; b < MB; ++b) red[wave][tt][b][lane] = acc[tt][b];
  __syncthreads();
  // D[i][j] of tile (tt, b): lane holds j = lane % 16 (activation row) and
  // i = 4 (lane / 16) + 0..3 (weight row) -> 4 consecutive output columns.
  if constexpr (EPI == 2) {
    for (int idx = threadIdx.x; idx < 2 * MB * 64; idx += 256) {
      const int l = idx & 63;
      const int tb = idx >> 6;
      const int tt = tb / MB, b = tb - (tb / MB) * MB;  // tt in {0, 1}: gate rows
      const f32x4 g = red[0][tt][b][l] + red[1][tt][b][l] + red[2][tt][b][l] + red[3][tt][b][l];
      const f32x4 u = red[0][tt + 2][b][l] + red[1][tt + 2][b][l] + red[2][tt + 2][b][l] +
                      red[3][tt + 2][b][l];
      const int m = m0 + 16 * b + (l & 15);
      const int j = j0 + 16 * tt + 4 * (l >> 4);
      if (m < M) {
        uint2 o;
        o.x = pack_bf16x2(g.x / (1.f + __expf(-g.x)) * u.x, g.y / (1.f + __expf(-g.y)) * u.y);
        o.y = pack_bf16x2(g.z / (1.f + __expf(-g.z)) * u.z, g.w / (1.f + __expf(-g.w)) * u.w);
        *reinterpret_cast<uint2*>(out_bf16 + (size_t)m * F + j) = o;
      }
    }
  } else {
    for (int idx = threadIdx.x; idx < 4 * MB * 64; idx += 256) {
      const int l = idx & 63;
      const int tb = idx >> 6;
      const int tt = tb / MB, b = tb - (tb / MB) * MB;
      const f32x4 v = red[0][tt][b][l] + red[1][tt][b][l] + red[2][tt][b][l] + red[3][tt][b][l];
      const int m = m0 + 16 * b + (l & 15);
      const int n = blockIdx.x * 64 + 16 * tt + 4 * (l >> 4);
      if (m < M) {
        f32x4* dst = reinterpret_cast<f32x4*>(out + (size_t)s * M * N + (size_t)m * N + n);
        if (accumulate) *dst = *dst + v;
        else *dst = v;
      }
    }
  }
}

// Sum split-K partials in split order and apply the epilogue (standalone
// sevo_linear with a split K range).
__global__ __launch_bounds__(256) void linear_epilogue_kernel(const float* __restrict__ part,
                                                              int S, int M, int N, int mode,
                                                              float* __restrict__ out_f32) {
  const size_t MN = (size_t)M * N;
  const size_t total4 = MN / 4;
  for (size_t g = (size_t)blockIdx.x * blockDim.x + threadIdx.x; g < total4;
       g += (size_t)gridDim.x * blockDim.x) {
    f32x4 a = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < S; ++s) a += *reinterpret_cast<const f32x4*>(part + s * MN + g * 4);
    f32x4* dst = reinterpret_cast<f32x4*>(out_f32 + g * 4);
    if (mode == 1) *dst = *dst + a;
    else *dst = a;
  }
}

LinearPlan plan_linear(int m, int n_out, int k, int k_splits, int mode) {
  LinearPlan p;
  if (mode == 2) {
    k_splits = 1;  // the SwiGLU product needs the whole K range
  } else if (k_splits <= 0) {
    // enough workgroups to keep the CUs streaming, but at least 1024 k
    // (16 steps) per workgroup so the pipeline has something to overlap
    const int tiles = (n_out / 64) * ((m + 63) / 64);
    int s = 1;
    while (tiles * s < 512 && k / (2 * s) >= 1024) s *= 2;
    k_splits = s;
  }
  int chunk = (k + k_splits - 1) / k_splits;
  chunk = (chunk + 127) / 128 * 128;
  p.k_chunk = chunk;
  p.k_splits = (k + chunk - 1) / chunk;
  return p;
}

size_t linear_workspace_bytes(int m, int n_out, int k, int k_splits, int mode) {
  const LinearPlan p = plan_linear(m, n_out, k, k_splits, mode);
  if (p.k_splits == 1) return 0;
  return (size_t)p.k_splits * m * n_out * sizeof(float);
}

template <int EPI>
static void launch_linear_kernel(int mb, dim3 grid, hipStream_t st, const bf16_t* x, int ldx,
                                 int m, const bf16_t* w, int n_out, int k, int k_chunk,
                                 float* dst, int acc, bf16_t* out_bf16) {
  if (mb == 4)
    hipLaunchKernelGGL((linear_kernel<4, EPI>), grid, dim3(256), 0, st, x, ldx, m, w, n_out, k,
                       k_chunk, dst, acc, out_bf16);
  else if (mb == 2)
    hipLaunchKernelGGL((linear_kernel<2, EPI>), grid, dim3(256), 0, st, x, ldx, m, w, n_out, k,
                       k_chunk, dst, acc, out_bf16);
  else
    hipLaunchKernelGGL((linear_kernel<1, EPI>), grid, dim3(256), 0, st, x, ldx, m, w, n_out, k,
                       k_chunk, dst, acc, out_bf16);
}

hipError_t launch_linear_partials(int m, int n_out, int k, int ldx, const LinearPlan& plan,
                                  const bf16_t* x, const bf16_t* w, float* out, int accumulate,
                                  hipStream_t st) {
  if (m == 0) return hipSuccess;
  const int mb = m > 32 ? 4 : (m > 16 ? 2 : 1);
  const dim3 grid(n_out / 64, plan.k_splits, m > 64 ? (m + 63) / 64 : 1);
  launch_linear_kernel<0>(m > 64 ? 4 : mb, grid, st, x, ldx, m, w, n_out, k, plan.k_chunk, out,
                          accumulate, nullptr);
  return hipGetLastError();
}

hipError_t launch_linear(int m, int n_out, int k, int ldx, int mode, const LinearPlan& plan,
                         const bf16_t* x, const bf16_t* w, void* out, float* workspace,
                         hipStream_t st) {
  if (m == 0) return hipSuccess;
  const int mb = m > 32 ? 4 : (m > 16 ? 2 : 1);
  const int zt = m > 64 ? (m + 63) / 64 : 1;
  if (mode == 2) {
    launch_linear_kernel<2>(m > 64 ? 4 : mb, dim3(n_out / 64, 1, zt), st, x, ldx, m, w, n_out, k,
                            plan.k_chunk, nullptr, 0, reinterpret_cast<bf16_t*>(out));
    return hipGetLastError();
  }
  if (plan.k_splits == 1)
    return launch_linear_partials(m, n_out, k, ldx, plan, x, w, reinterpret_cast<float*>(out),
                                  mode == 1 ? 1 : 0, st);
  hipError_t e = launch_linear_partials(m, n_out, k, ldx, plan, x, w, workspace, 0, st);
  if (e != hipSuccess) return e;
  const size_t total4 = (size_t)m * n_out / 4;
  size_t blocks = (total4 + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(linear_epilogue_kernel, dim3((unsigned)blocks), dim3(256), 0, st, workspace,
                     plan.k_splits, m, n_out, mode, reinterpret_cast<float*>(out));
  return hipGetLastError();
}

}  // namespace sevo
