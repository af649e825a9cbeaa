// Skinny bf16 GEMM Y = X W^T on the gfx950 matrix cores, for the QKV, output,
// gate/up and down projections and the LM head of a decode step.
//
// At decode the batch M is the population size (<= 64 per tile), so the
// arithmetic intensity is M flop per weight byte: far below the MFMA ridge,
// the kernel is a weight stream and is designed for HBM bandwidth.
//   * operands are stored fragment-major (common.h): every load of an MFMA
//     16x16x32 operand fragment is one contiguous 1 KB read (half-line reads
//     of row-major rows measured about a third slower);
//   * one 256-thread workgroup per (RB row blocks of 16 weight rows, K split,
//     M tile of up to 64 rows).  The planner picks RB and the split count so
//     that a projection is about one round of 256 equal workgroups, one per
//     CU (a 384-workgroup gate/up or a 192-workgroup QKV left CUs with half
//     or double the bytes of the others); more row blocks per workgroup also
//     share each activation fragment among more weight fragments;
//   * the four waves take the 32-k steps of the split round-robin (wave w:
//     steps w, w + 4, ...); at a step a wave loads RB weight fragments and
//     the M tile's activation fragments and runs RB x MB MFMAs;
//   * weights are loaded non-temporally: they are read once, and without the
//     hint their stream evicts the activation fragments, which every
//     workgroup re-reads, from L2 (cached activations and streamed weights
//     measured 2-11% faster per projection);
//   * A operand = 16 weight rows x 32 k, B operand = 16 activation rows x 32 k;
//   * four register fragment buffers keep the next three steps' loads in
//     flight while the current step's MFMAs run;
//   * the four waves' fp32 tiles are summed through LDS.  With K split across
//     workgroups the fp32 partials [split][m][n] are summed, in split order, by
//     the consumer (the epilogue kernel here, or the fused norm / RoPE kernels
//     of the decode step).  The SwiGLU form takes gate/up pairs: the packed
//     superblock holds 32 gate rows followed by the matching 32 up rows, so
//     row blocks (h, h + 2) of superblock s are gate and up of output columns
//     32 s + 16 h .. + 15, and it writes silu(g) * u.
#include "common.h"
#include "kernels.h"

namespace sevo {

template <int MB, int RB>
struct GemmFrag {
  bf16x8v a[RB];
  bf16x8v b[MB];
};

// Registers: four fragment buffers of RB + MB fragments (4 VGPRs each) plus
// RB x MB accumulators; two workgroups per CU while that fits in 256.
template <int MB, int RB>
constexpr int linear_min_blocks() {
  return 16 * (RB + MB) + 4 * RB * MB + 24 <= 256 ? 2 : 1;
}

// EPI 0: fp32 tile (split partial, or final with optional accumulate)
// EPI 2: SwiGLU, bf16 out[m][F] (row-major or tiled; needs the full K range)
// XT: X in the tiled activation layout (else row-major with stride ldx)
template <int MB, int RB, int EPI, int XT>
__global__ __launch_bounds__(256, (linear_min_blocks<MB, RB>())) void linear_kernel(
    const bf16_t* __restrict__ X, int ldx, int M, const bf16_t* __restrict__ W, int N, int K,
    int k_chunk, float* __restrict__ out, int accumulate, bf16_t* __restrict__ out_bf16,
    int out_tiled) {
  static_assert(EPI != 2 || RB % 2 == 0, "SwiGLU row blocks come in gate/up pairs");
  __shared__ f32x4 red[4][RB][MB][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int s = blockIdx.y;
  const int m0 = blockIdx.z * 16 * MB;
  const int r = lane & 15, q = lane >> 4;
  const int KS = K >> 5;
  const int nrb = N >> 4;

  // row block i of this workgroup: fragment tt of superblock sb, at
  // W + woff[i] + st * 2048 for step st.  Row blocks past the matrix read
  // superblock 0 and are never stored.
  size_t woff[RB];
#pragma unroll
  for (int i = 0; i < RB; ++i) {
    int sb, tt;
    if constexpr (EPI == 2) {
      const int p = blockIdx.x * (RB / 2) + (i >> 1);  // gate/up pair
      sb = p >> 1;
      tt = (p & 1) + 2 * (i & 1);
      if (2 * p >= nrb) sb = tt = 0;
    } else {
      const int rbk = blockIdx.x * RB + i;
      sb = rbk >> 2;
      tt = rbk & 3;
      if (rbk >= nrb) sb = tt = 0;
    }
    woff[i] = ((size_t)sb * KS * 4 + tt) * 512 + lane * 8;
  }
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

  f32x4 acc[RB][MB];
#pragma unroll
  for (int i = 0; i < RB; ++i)
#pragma unroll
    for (int b = 0; b < MB; ++b) acc[i][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  // j-th step of this wave; past the end it re-reads the last one (L2 hits)
  auto load = [&](GemmFrag<MB, RB>& f, int j) {
    const int st = st_base + wave + 4 * min(j, cnt - 1);
#pragma unroll
    for (int i = 0; i < RB; ++i)
      f.a[i] = __builtin_nontemporal_load(
          reinterpret_cast<const bf16x8v*>(W + woff[i] + (size_t)st * 2048));
#pragma unroll
    for (int b = 0; b < MB; ++b)
      f.b[b] = *reinterpret_cast<const bf16x8v*>(xp[b] + (XT ? (size_t)st * 512 : (size_t)st * 32));
  };
  auto mma = [&](const GemmFrag<MB, RB>& f) {
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
      for (int b = 0; b < MB; ++b)
        acc[i][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.a[i], f.b[b], acc[i][b], 0, 0, 0);
  };

  // Four fragment buffers rotate four steps per trip: while one is
  // multiplied the next three are in flight.  sched_barrier keeps the
  // scheduler from sinking the prefetch loads next to their MFMAs, which
  // would serialise the stream.  The step-count tests are wave-uniform.
  if (cnt > 0) {
    GemmFrag<MB, RB> f0, f1, f2, f3;
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
  for (int i = 0; i < RB; ++i)
#pragma unroll
    for (int b = 0; b < MB; ++b) red[wave][i][b][lane] = acc[i][b];
  __syncthreads();
  // D[i][j] of tile (row block, b): lane holds j = lane % 16 (activation row)
  // and i = 4 (lane / 16) + 0..3 (weight row) -> 4 consecutive output columns.
  if constexpr (EPI == 2) {
    const int F = N / 2;
    for (int idx = threadIdx.x; idx < (RB / 2) * MB * 64; idx += 256) {
      const int l = idx & 63;
      const int tb = idx >> 6;
      const int pi = tb / MB, b = tb - pi * MB;
      const int p = blockIdx.x * (RB / 2) + pi;
      const int gi = 2 * pi, ui = 2 * pi + 1;
      const f32x4 g = red[0][gi][b][l] + red[1][gi][b][l] + red[2][gi][b][l] + red[3][gi][b][l];
      const f32x4 u = red[0][ui][b][l] + red[1][ui][b][l] + red[2][ui][b][l] + red[3][ui][b][l];
      const int m = m0 + 16 * b + (l & 15);
      const int j = (p >> 1) * 32 + 16 * (p & 1) + 4 * (l >> 4);
      if (m < M && 2 * p < nrb) {
        uint2 o;
        o.x = pack_bf16x2(g.x / (1.f + __expf(-g.x)) * u.x, g.y / (1.f + __expf(-g.y)) * u.y);
        o.y = pack_bf16x2(g.z / (1.f + __expf(-g.z)) * u.z, g.w / (1.f + __expf(-g.w)) * u.w);
        const size_t off = out_tiled ? act_tile_offset(m, j, F) : (size_t)m * F + j;
        *reinterpret_cast<uint2*>(out_bf16 + off) = o;
      }
    }
  } else {
    for (int idx = threadIdx.x; idx < RB * MB * 64; idx += 256) {
      const int l = idx & 63;
      const int tb = idx >> 6;
      const int i = tb / MB, b = tb - i * MB;
      const f32x4 v = red[0][i][b][l] + red[1][i][b][l] + red[2][i][b][l] + red[3][i][b][l];
      const int m = m0 + 16 * b + (l & 15);
      const int rbk = blockIdx.x * RB + i;
      const int n = rbk * 16 + 4 * (l >> 4);
      if (m < M && rbk < nrb) {
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
    for (int s0 = 0; s0 < S; s0 += 4) {  // split order; four splits' loads together
      f32x4 p[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (s0 + j < S) p[j] = *reinterpret_cast<const f32x4*>(part + (s0 + j) * MN + g * 4);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (s0 + j < S) a += p[j];
    }
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

static int pick_mb(int m) { return m > 32 ? 4 : (m > 16 ? 2 : 1); }

// Row blocks per workgroup with an instantiated kernel: at least 3 for a
// 64-row M tile (fewer re-read each activation fragment for too few weight
// fragments), at most what the registers hold; SwiGLU takes whole pairs.
static int rb_min(int mb) { return mb == 4 ? 3 : 2; }
static int rb_max(int mb) { return mb == 4 ? 8 : (mb == 2 ? 12 : 16); }
static const int kRbSet[] = {2, 3, 4, 5, 6, 8, 10, 12, 14, 16};
static bool rb_ok(int rb, int mb, int swiglu) {
  return rb >= rb_min(mb) && rb <= rb_max(mb) && (!swiglu || rb % 2 == 0);
}

LinearPlan plan_linear(int m, int n_out, int k, int k_splits, int mode) {
  const int mb = pick_mb(m);
  const int mt = (m + 16 * mb - 1) / (16 * mb);
  const int swiglu = mode == 2;
  const int per_unit = swiglu ? 2 : 1;  // row blocks per unit (a gate/up pair)
  const int units = (n_out / 16) / per_unit;
  auto chunk_of = [&](int s) {
    const int c = (k + s - 1) / s;
    return (c + 127) / 128 * 128;
  };
  // workgroups of a plan, and the share of the CUs its last round keeps busy
  // (one workgroup per CU per round)
  auto wgs_of = [&](int rb, int s) {
    const int upw = rb / per_unit;
    return ((units + upw - 1) / upw) * s * mt;
  };
  auto eff_of = [&](int wgs) { return wgs / (double)(((wgs + 255) / 256) * 256); };
  // the row-block count for split count s: the fewest that fit the
  // projection in one round of 256 workgroups; past the register limit
  // (several rounds) the one whose rounds are fullest, the larger on near ties
  auto rb_for = [&](int s) {
    const long need = ((long)units * s * mt + 255) / 256 * per_unit;
    for (int rb : kRbSet)
      if (rb >= need && rb_ok(rb, mb, swiglu)) return rb;
    int best = 0;
    double best_eff = -1.0;
    for (int rb : kRbSet) {
      if (!rb_ok(rb, mb, swiglu) || 2 * rb < rb_max(mb)) continue;
      const double e = eff_of(wgs_of(rb, s));
      if (e > best_eff - 0.01) {
        if (e > best_eff) best_eff = e;
        best = rb;
      }
    }
    return best;
  };
  LinearPlan p;
  // split counts: SwiGLU needs the whole K range; otherwise the caller's, or
  // the smallest of 1, 2, 4, ... (at least 1024 k per split, so each wave
  // streams 8 steps or more) whose plan fills 95% of its last round or needs
  // more than one round, else the fullest.  Split partials cost M x n_out x 8 bytes each (written and
  // read back), so more splits must fill the rounds clearly better (by 2%).
  // A projection too small for 64 workgroups even at 1024 k per split (a MoE
  // router: 128 experts) may split down to 256 k; its partials are tiny.
  int cands[5], nc = 0;
  const int upw_min = (rb_min(mb) + per_unit - 1) / per_unit;
  const long wgs_1024 = (long)((units + upw_min - 1) / upw_min) * mt * (k >= 2048 ? k / 1024 : 1);
  const int min_chunk = wgs_1024 < 64 ? 256 : 1024;
  if (swiglu) cands[nc++] = 1;
  else if (k_splits > 0) cands[nc++] = k_splits;
  else
    for (int s = 1; s <= 16; s *= 2)
      if (s == 1 || chunk_of(s) >= min_chunk) cands[nc++] = s;
  double best_eff = -1.0;
  for (int i = 0; i < nc; ++i) {
    const int chunk = chunk_of(cands[i]);
    const int s = (k + chunk - 1) / chunk;
    const int rb = rb_for(s);
    const int wgs = wgs_of(rb, s);
    const double e = eff_of(wgs);
    if (e > best_eff + 0.02) {
      best_eff = e;
      p.k_chunk = chunk;
      p.k_splits = s;
      p.rb = rb;
    }
    if (e >= 0.95 || wgs > 256) break;
  }
  return p;
}

size_t linear_workspace_bytes(int m, int n_out, int k, int k_splits, int mode) {
  const LinearPlan p = plan_linear(m, n_out, k, k_splits, mode);
  if (p.k_splits == 1) return 0;
  return (size_t)p.k_splits * m * n_out * sizeof(float);
}

struct LinearLaunch {
  dim3 grid;
  hipStream_t st;
  const bf16_t* x;
  int ldx, m;
  const bf16_t* w;
  int n_out, k, k_chunk;
  float* dst;
  int acc;
  bf16_t* out_bf16;
  int out_tiled;
};

template <int MB, int RB, int EPI, int XT>
static bool launch_one(const LinearLaunch& a) {
  constexpr bool inst = RB >= (MB == 4 ? 3 : 2) && RB <= (MB == 4 ? 8 : (MB == 2 ? 12 : 16)) &&
                        (EPI != 2 || RB % 2 == 0);
  if constexpr (inst) {
    hipLaunchKernelGGL((linear_kernel<MB, RB, EPI, XT>), a.grid, dim3(256), 0, a.st, a.x, a.ldx,
                       a.m, a.w, a.n_out, a.k, a.k_chunk, a.dst, a.acc, a.out_bf16, a.out_tiled);
    return true;
  } else {
    return false;
  }
}

template <int MB, int EPI, int XT>
static bool launch_rb(int rb, const LinearLaunch& a) {
  switch (rb) {
    case 2: return launch_one<MB, 2, EPI, XT>(a);
    case 3: return launch_one<MB, 3, EPI, XT>(a);
    case 4: return launch_one<MB, 4, EPI, XT>(a);
    case 5: return launch_one<MB, 5, EPI, XT>(a);
    case 6: return launch_one<MB, 6, EPI, XT>(a);
    case 8: return launch_one<MB, 8, EPI, XT>(a);
    case 10: return launch_one<MB, 10, EPI, XT>(a);
    case 12: return launch_one<MB, 12, EPI, XT>(a);
    case 14: return launch_one<MB, 14, EPI, XT>(a);
    case 16: return launch_one<MB, 16, EPI, XT>(a);
    default: return false;
  }
}

template <int EPI, int XT>
static hipError_t launch_linear_kernel(int mb, int rb, const LinearLaunch& a) {
  bool ok;
  if (mb == 4) ok = launch_rb<4, EPI, XT>(rb, a);
  else if (mb == 2) ok = launch_rb<2, EPI, XT>(rb, a);
  else ok = launch_rb<1, EPI, XT>(rb, a);
  return ok ? hipGetLastError() : hipErrorInvalidValue;
}

static dim3 linear_grid(int m, int n_out, int mode, const LinearPlan& plan) {
  const int mb = pick_mb(m);
  const int per_unit = mode == 2 ? 2 : 1;
  const int units = (n_out / 16) / per_unit;
  const int upw = plan.rb / per_unit;
  return dim3((units + upw - 1) / upw, mode == 2 ? 1 : plan.k_splits,
              (m + 16 * mb - 1) / (16 * mb));
}

hipError_t launch_linear_partials(int m, int n_out, int k, int ldx, int x_tiled,
                                  const LinearPlan& plan, const bf16_t* x, const bf16_t* w,
                                  float* out, int accumulate, hipStream_t st) {
  if (m == 0) return hipSuccess;
  const LinearLaunch a{linear_grid(m, n_out, 0, plan), st, x, ldx, m, w, n_out, k, plan.k_chunk,
                       out, accumulate, nullptr, 0};
  return x_tiled ? launch_linear_kernel<0, 1>(pick_mb(m), plan.rb, a)
                 : launch_linear_kernel<0, 0>(pick_mb(m), plan.rb, a);
}

hipError_t launch_linear(int m, int n_out, int k, int ldx, int x_tiled, int mode,
                         const LinearPlan& plan, const bf16_t* x, const bf16_t* w, void* out,
                         int out_tiled, float* workspace, hipStream_t st) {
  if (m == 0) return hipSuccess;
  if (mode == 2) {
    const LinearLaunch a{linear_grid(m, n_out, 2, plan), st, x, ldx, m, w, n_out, k,
                         plan.k_chunk, nullptr, 0, reinterpret_cast<bf16_t*>(out), out_tiled};
    return x_tiled ? launch_linear_kernel<2, 1>(pick_mb(m), plan.rb, a)
                   : launch_linear_kernel<2, 0>(pick_mb(m), plan.rb, a);
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
