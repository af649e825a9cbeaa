// Skinny bf16 GEMM Y = X W^T on the gfx950 matrix cores, for the QKV, output,
// gate/up and down projections and the LM head of a decode step.
//
// At decode the batch M is the population size (<= 64 per tile), so the
// arithmetic intensity is M flop per weight byte: far below the MFMA ridge,
// the kernel is a weight stream and is designed for HBM bandwidth.
//   * operands are stored fragment-major (common.h): every load of an MFMA
//     16x16x32 operand fragment is one contiguous 1 KB read (half-line reads
//     of row-major rows measured about a third slower);
//   * one 256-thread workgroup per (64-row weight superblock, K split,
//     64-row M tile); the packed layout makes the superblock one contiguous
//     region, read front to back;
//   * the four waves take the 32-k steps of the split round-robin (wave w:
//     steps w, w + 4, ...), so at any time the workgroup reads one contiguous
//     window of the region;
//   * A operand = 16 weight rows x 32 k, B operand = 16 activation rows x 32 k
//     (the activations are tiny and stay in L2);
//   * four register fragment buffers keep the next three steps' loads in
//     flight while the current step's MFMAs run;
//   * the four waves' fp32 tiles are summed through LDS.  With K split across
//     workgroups the fp32 partials [split][m][n] are summed, in split order, by
//     the consumer (the epilogue kernel here, or the fused norm / RoPE kernels
//     of the decode step).  The SwiGLU form reads a superblock packed as 32
//     gate rows followed by the matching 32 up rows and writes silu(g) * u.
#include "common.h"
#include "kernels.h"

namespace sevo {

template <int MB>
struct GemmFrag {
  bf16x8v a[4];
  bf16x8v b[MB];
};

// EPI 0: fp32 tile (split partial, or final with optional accumulate)
// EPI 2: SwiGLU, bf16 out[m][F] (row-major or tiled; needs the full K range)
// XT: X in the tiled activation layout (else row-major with stride ldx)
template <int MB, int EPI, int XT>
__global__ __launch_bounds__(256, 2) void linear_kernel(const bf16_t* __restrict__ X, int ldx,
                                                        int M, const bf16_t* __restrict__ W, int N,
                                                        int K, int k_chunk, float* __restrict__ out,
                                                        int accumulate,
                                                        bf16_t* __restrict__ out_bf16,
                                                        int out_tiled) {
  __shared__ f32x4 red[4][4][MB][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int sb = blockIdx.x;
  const int s = blockIdx.y;
  const int m0 = blockIdx.z * 16 * MB;
  const int r = lane & 15, q = lane >> 4;
  const int KS = K >> 5;

  // weight fragment (step st, row block tt) at wp + st * 2048 + tt * 512
  const bf16_t* wp = W + (size_t)sb * KS * 2048 + lane * 8;
  // activation rows past M read the last valid row (block): they only feed
  // output rows that are never stored, so no masking is needed
  const bf16_t* xp[MB];
#pragma unroll
  for (int b = 0; b < MB; ++b) {
    if constexpr (XT) {
      const int blk = min((m0 >> 4) + b, (M - 1) >> 4);
      xp[b] = X + (size_t)blk * KS * 512 + lane * 8;
    } else {
      const int row = min(m0 + 16 * b + r, M - 1);
      xp[b] = X + (size_t)row * ldx + 8 * q;
    }
  }

  const int kb = s * k_chunk;
  const int ke = min(K, kb + k_chunk);
  const int st_base = kb >> 5;
  const int nsteps = (ke - kb) >> 5;
  const int cnt = nsteps > wave ? (nsteps - wave + 3) >> 2 : 0;  // steps of this wave

  f32x4 acc[4][MB];
#pragma unroll
  for (int tt = 0; tt < 4; ++tt)
#pragma unroll
    for (int b = 0; b < MB; ++b) acc[tt][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  // j-th step of this wave; past the end it re-reads the last one (L2 hits)
  auto load = [&](GemmFrag<MB>& f, int j) {
    const int st = st_base + wave + 4 * min(j, cnt - 1);
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
      f.a[tt] = *reinterpret_cast<const bf16x8v*>(wp + (size_t)st * 2048 + tt * 512);
#pragma unroll
    for (int b = 0; b < MB; ++b)
      f.b[b] = *reinterpret_cast<const bf16x8v*>(xp[b] + (XT ? (size_t)st * 512 : (size_t)st * 32));
  };
  auto mma = [&](const GemmFrag<MB>& f) {
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
      for (int b = 0; b < MB; ++b)
        acc[tt][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.a[tt], f.b[b], acc[tt][b], 0, 0, 0);
  };

  // Four fragment buffers rotate four steps per trip: while one is
  // multiplied the next three are in flight.  sched_barrier keeps the
  // scheduler from sinking the prefetch loads next to their MFMAs, which
  // would serialise the stream.  The step-count tests are wave-uniform.
  if (cnt > 0) {
    GemmFrag<MB> f0, f1, f2, f3;
    load(f0, 0);
    load(f1, 1);
    load(f2, 2);
    for (int j = 0; j < cnt; j += 4) {
      load(f3, j + 3);
      __builtin_amdgcn_sched_barrier(0);
      mma(f0);
      __builtin_amdgcn_sched_barrier(0);
      load(f0, j + 4);
      __builtin_amdgcn_sched_barrier(0);
      if (j + 1 < cnt) mma(f1);
      __builtin_amdgcn_sched_barrier(0);
      load(f1, j + 5);
      __builtin_amdgcn_sched_barrier(0);
      if (j + 2 < cnt) mma(f2);
      __builtin_amdgcn_sched_barrier(0);
      load(f2, j + 6);
      __builtin_amdgcn_sched_barrier(0);
      if (j + 3 < cnt) mma(f3);
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
    const int F = N / 2;
    for (int idx = threadIdx.x; idx < 2 * MB * 64; idx += 256) {
      const int l = idx & 63;
      const int tb = idx >> 6;
      const int tt = tb / MB, b = tb - (tb / MB) * MB;  // tt in {0, 1}: gate rows
      const f32x4 g = red[0][tt][b][l] + red[1][tt][b][l] + red[2][tt][b][l] + red[3][tt][b][l];
      const f32x4 u = red[0][tt + 2][b][l] + red[1][tt + 2][b][l] + red[2][tt + 2][b][l] +
                      red[3][tt + 2][b][l];
      const int m = m0 + 16 * b + (l & 15);
      const int j = sb * 32 + 16 * tt + 4 * (l >> 4);
      if (m < M) {
        uint2 o;
        o.x = pack_bf16x2(g.x / (1.f + __expf(-g.x)) * u.x, g.y / (1.f + __expf(-g.y)) * u.y);
        o.y = pack_bf16x2(g.z / (1.f + __expf(-g.z)) * u.z, g.w / (1.f + __expf(-g.w)) * u.w);
        const size_t off = out_tiled ? act_tile_offset(m, j, F) : (size_t)m * F + j;
        *reinterpret_cast<uint2*>(out_bf16 + off) = o;
      }
    }
  } else {
    for (int idx = threadIdx.x; idx < 4 * MB * 64; idx += 256) {
      const int l = idx & 63;
      const int tb = idx >> 6;
      const int tt = tb / MB, b = tb - (tb / MB) * MB;
      const f32x4 v = red[0][tt][b][l] + red[1][tt][b][l] + red[2][tt][b][l] + red[3][tt][b][l];
      const int m = m0 + 16 * b + (l & 15);
      const int n = sb * 64 + 16 * tt + 4 * (l >> 4);
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

// Row-major [N][K] -> packed layout, one thread per 8-element run of dst.
__global__ __launch_bounds__(256) void pack_weight_kernel(const bf16_t* __restrict__ src,
                                                          bf16_t* __restrict__ dst, int N, int K,
                                                          int gate_up) {
  const size_t runs = (size_t)N * K / 8;
  const int KS = K >> 5;
  for (size_t g = (size_t)blockIdx.x * blockDim.x + threadIdx.x; g < runs;
       g += (size_t)gridDim.x * blockDim.x) {
    const size_t e = g * 8;
    const size_t blk = e >> 11;  // (superblock, step)
    const int rem = (int)(e & 2047);
    const int tt = rem >> 9;
    const int ln = (rem & 511) >> 3;
    const int sbk = (int)(blk / KS);
    const int st = (int)(blk - (size_t)sbk * KS);
    int row;
    if (gate_up) row = (tt < 2 ? 0 : N / 2) + sbk * 32 + (tt & 1) * 16 + (ln & 15);
    else row = sbk * 64 + tt * 16 + (ln & 15);
    const int col = st * 32 + (ln >> 4) * 8;
    *reinterpret_cast<u32x4*>(dst + e) =
        *reinterpret_cast<const u32x4*>(src + (size_t)row * K + col);
  }
}

LinearPlan plan_linear(int m, int n_out, int k, int k_splits, int mode) {
  LinearPlan p;
  if (mode == 2) {
    k_splits = 1;  // the SwiGLU product needs the whole K range
  } else if (k_splits <= 0) {
    // about 192 or more workgroups (superblocks x M tiles x splits) so the
    // CUs are busy, but at least 1024 k (8 steps per wave) per split so each
    // wave streams a while; split partials cost M x n_out x 8 bytes each
    const int tiles = (n_out / 64) * ((m + 63) / 64);
    int s = 1;
    while (tiles * s < 192 && k / (2 * s) >= 1024) s *= 2;
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

template <int EPI, int XT>
static void launch_linear_kernel(int mb, dim3 grid, hipStream_t st, const bf16_t* x, int ldx,
                                 int m, const bf16_t* w, int n_out, int k, int k_chunk,
                                 float* dst, int acc, bf16_t* out_bf16, int out_tiled) {
  if (mb == 4)
    hipLaunchKernelGGL((linear_kernel<4, EPI, XT>), grid, dim3(256), 0, st, x, ldx, m, w, n_out,
                       k, k_chunk, dst, acc, out_bf16, out_tiled);
  else if (mb == 2)
    hipLaunchKernelGGL((linear_kernel<2, EPI, XT>), grid, dim3(256), 0, st, x, ldx, m, w, n_out,
                       k, k_chunk, dst, acc, out_bf16, out_tiled);
  else
    hipLaunchKernelGGL((linear_kernel<1, EPI, XT>), grid, dim3(256), 0, st, x, ldx, m, w, n_out,
                       k, k_chunk, dst, acc, out_bf16, out_tiled);
}

static int pick_mb(int m) { return m > 32 ? 4 : (m > 16 ? 2 : 1); }

hipError_t launch_linear_partials(int m, int n_out, int k, int ldx, int x_tiled,
                                  const LinearPlan& plan, const bf16_t* x, const bf16_t* w,
                                  float* out, int accumulate, hipStream_t st) {
  if (m == 0) return hipSuccess;
  const int mb = pick_mb(m);
  const dim3 grid(n_out / 64, plan.k_splits, (m + 16 * mb - 1) / (16 * mb));
  if (x_tiled)
    launch_linear_kernel<0, 1>(mb, grid, st, x, ldx, m, w, n_out, k, plan.k_chunk, out,
                               accumulate, nullptr, 0);
  else
    launch_linear_kernel<0, 0>(mb, grid, st, x, ldx, m, w, n_out, k, plan.k_chunk, out,
                               accumulate, nullptr, 0);
  return hipGetLastError();
}

hipError_t launch_linear(int m, int n_out, int k, int ldx, int x_tiled, int mode,
                         const LinearPlan& plan, const bf16_t* x, const bf16_t* w, void* out,
                         int out_tiled, float* workspace, hipStream_t st) {
  if (m == 0) return hipSuccess;
  if (mode == 2) {
    const int mb = pick_mb(m);
    const dim3 grid(n_out / 64, 1, (m + 16 * mb - 1) / (16 * mb));
    bf16_t* o = reinterpret_cast<bf16_t*>(out);
    if (x_tiled)
      launch_linear_kernel<2, 1>(mb, grid, st, x, ldx, m, w, n_out, k, plan.k_chunk, nullptr, 0,
                                 o, out_tiled);
    else
      launch_linear_kernel<2, 0>(mb, grid, st, x, ldx, m, w, n_out, k, plan.k_chunk, nullptr, 0,
                                 o, out_tiled);
    return hipGetLastError();
  }
  if (plan.k_splits == 1)
    return launch_linear_partials(m, n_out, k, ldx, x_tiled, plan, x, w,
                                  reinterpret_cast<float*>(out), mode == 1 ? 1 : 0, st);
  hipError_t e = launch_linear_partials(m, n_out, k, ldx, x_tiled, plan, x, w, workspace, 0, st);
  if (e != hipSuccess) return e;
  const size_t total4 = (size_t)m * n_out / 4;
  size_t blocks = (total4 + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(linear_epilogue_kernel, dim3((unsigned)blocks), dim3(256), 0, st, workspace,
                     plan.k_splits, m, n_out, mode, reinterpret_cast<float*>(out));
  return hipGetLastError();
}

hipError_t launch_pack_weight(const bf16_t* src, bf16_t* dst, int n_out, int k, int gate_up,
                              hipStream_t st) {
  const size_t runs = (size_t)n_out * k / 8;
  if (runs == 0) return hipSuccess;
  size_t blocks = (runs + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  hipLaunchKernelGGL(pack_weight_kernel, dim3((unsigned)blocks), dim3(256), 0, st, src, dst,
                     n_out, k, gate_up);
  return hipGetLastError();
}

}  // namespace sevo
