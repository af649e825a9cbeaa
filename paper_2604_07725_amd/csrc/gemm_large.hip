// Large-M bf16 GEMM Y = X W^T on the gfx950 matrix cores: the projections of
// a prefill (the confidence engine's scoring pass), where M is a token count
// in the thousands and the product is compute-bound (intensity ~ M flop per
// weight byte, far above the ~315 flop/byte ridge of the chip).
//
//   * workgroup tile 256 (m) x 256 (n), 8 waves in a 2 x 4 grid, each wave a
//     128 x 64 sub-tile held as 4 x 2 accumulators of the 32x32x16 bf16 MFMA
//     (128 fp32 per lane, 180 registers in all), so two waves share each SIMD
//     and one issues MFMAs while the other waits on its LDS reads or a
//     barrier (2-3% faster than 4 waves of 128 x 128 sub-tiles, one per
//     SIMD, on every 8B-class shape at M = 16K and 40K);
//   * K is consumed in stages of 32: the 16 KB X slice and the 16 KB W slice
//     of a stage go straight from global memory into LDS with the gfx950
//     direct-to-LDS loads (16 bytes per lane, no register staging); four LDS
//     stages (128 KB) keep three stages of loads in flight under the MFMAs;
//   * both operands keep the fragment-major layouts of the decode path (the
//     packed weights and the tiled activations, 1 KB per 16 x 32 fragment), so
//     every direct load is one contiguous 1 KB per wave and every LDS read of
//     a 16-lane group is 256 contiguous bytes (no bank conflicts, no swizzle);
//     a row-major X is gathered into the same LDS order by the per-lane
//     addresses of the direct loads;
//   * the tile order is XCD-aware: consecutive workgroups land on different
//     XCDs, so the linear id is remapped to give each XCD a contiguous range
//     of tiles, walked in groups of 4 m-tiles so the X and W slices a group
//     streams are shared in that XCD's L2 (groups of 4 measured 1-4% faster
//     than 8 at M = 16K-40K, groups of 16 7-10% slower).
// Epilogues: fp32 store, fp32 accumulate (residual update), and SwiGLU over a
// gate/up matrix packed in 32 + 32 row superblocks (bf16 output, tiled or
// row-major).
//
// Grouped form (the mixture of experts of a prefill): the m-tiles are 256-entry
// tiles of the experts' entry lists (tile_off from the planner), a tile's
// weights are its expert's, and its A rows are gathered per lane: the entry's
// token row of the tiled normed input (gate/up), or the expert's SwiGLU rows
// (down).  The gate/up epilogue writes SwiGLU rows at the entries' positions;
// the down epilogue scatters routing weight * product into the per-slot
// outputs [slot][token][hidden].
#include "common.h"
#include "kernels.h"

namespace sevo {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kLgBM = 256, kLgBN = 256, kLgBK = 32, kLgStages = 4;
// one stage = one 32-column step: A 16 row blocks + B 4 superblocks x 4 fragments
constexpr int kLgStageElems = 16 * 512 + 16 * 512;
constexpr int kLgDmaPerStage = 4;  // direct loads per wave per stage
constexpr int kLgWaves = 8;

// EPI 0: out fp32 [M][ldo] = Y;  EPI 1: out += Y;  EPI 2: SwiGLU -> out_bf16;
// EPI 3 (grouped down): out [slot][token][N] = weight * Y
// XT 1: X in the tiled activation layout, else row-major with stride ldx
// GR 1: grouped (M = the rows of X: tokens for gate/up, entries for down)
template <int EPI, int XT, int GR>
__global__ __launch_bounds__(64 * kLgWaves, 1) void gemm_large_kernel(
    const bf16_t* __restrict__ X, int ldx, int M, const bf16_t* __restrict__ W, int N, int K,
    float* __restrict__ out, int ldo, bf16_t* __restrict__ out_bf16, int out_tiled, int tiles_m,
    int tiles_n, GroupArgs g) {
  __shared__ __attribute__((aligned(1024))) bf16_t smem[kLgStages * kLgStageElems];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 2, wn = wave & 3;

  // ---- tile order: XCD-contiguous ranges, groups of GM m-tiles
  const int total = tiles_m * tiles_n;
  int t = blockIdx.x;
  {
    const int per = total >> 3;  // full rounds of 8
    if (t < per * 8) t = (t & 7) * per + (t >> 3);
  }
  constexpr int GM = 4;
  const int group = t / (GM * tiles_n);
  const int first_m = group * GM;
  const int gsize = min(GM, tiles_m - first_m);
  const int in_group = t - group * GM * tiles_n;
  const int tm = first_m + in_group % gsize;
  const int tn = in_group / gsize;
  int m0 = tm * kLgBM;
  const int n0 = tn * kLgBN;
  // grouped: the expert of m-tile tm and the tile's first entry of that expert
  int rows = M;      // rows of this tile's matrix (the expert's entries)
  int ent0 = 0;      // first entry of the expert
  if constexpr (GR) {
    const int total_m = g.tile_off[g.E];
    if (tm >= total_m) return;  // uniform over the workgroup, before any barrier
    int lo = 0, hi = g.E;       // tile_off[lo] <= tm < tile_off[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (g.tile_off[mid] <= tm) lo = mid;
      else hi = mid;
    }
    ent0 = g.offsets[lo];
    rows = g.offsets[lo + 1] - ent0;
    m0 = (tm - g.tile_off[lo]) * kLgBM;
    W += (size_t)lo * N * K;
  }

  const int KS = K >> 5;  // 32-column steps = stages
  const int last_blk = (M - 1) >> 4;
  const int last_sb = (N >> 6) - 1;

  // ---- this wave's direct loads per stage: A row blocks 2w, 2w + 1 and
  // fragments 2 (w % 2), + 1 of B superblock w / 2, each through a wave-uniform descriptor
  // over the region it streams (byte offsets stay far below 2^32)
  __amdgpu_buffer_rsrc_t ra[2];
  uint32_t a_voff;  // this lane's byte offset at step 0 (plus 1 KB or 64 B per step)
  uint32_t g_voff[2];  // grouped: per-lane gathered row offsets (one descriptor)
  if constexpr (GR) {
    // one descriptor over the whole X; a row past the tile's entries gets an
    // offset past the records (the direct load then writes zeros)
    const uint32_t recs = XT ? (uint32_t)(((M + 15) >> 4) * 16) * K * 2 : (uint32_t)M * ldx * 2;
    ra[0] = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(X), 0, recs, 0x00020000);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int j = m0 + 16 * (2 * wave + i) + (lane & 15);
      g_voff[i] = 0x80000000u;
      if (j < rows) {
        if constexpr (XT) {
          const int tok = g.assign[ent0 + j] / g.k;
          g_voff[i] = (uint32_t)(((tok >> 4) * KS * 512 + (16 * (lane >> 4) + (tok & 15)) * 8) * 2);
        } else {
          g_voff[i] = (uint32_t)(((size_t)(ent0 + j) * ldx + 8 * (lane >> 4)) * 2);
        }
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 2 && !GR; ++i) {
    const int blk = min((m0 >> 4) + 2 * wave + i, last_blk);
    if constexpr (XT) {
      ra[i] = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(X + (size_t)blk * KS * 512), 0,
                                                KS * 1024, 0x00020000);
    } else {
      // run p = lane of the fragment is row 16 blk + p % 16, columns
      // 8 (p / 16) .. + 8 of the step; rows past M fall outside the records
      const int rows = min(16, M - 16 * blk);
      ra[i] = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(X + (size_t)16 * blk * ldx), 0,
                                                rows * ldx * 2, 0x00020000);
    }
  }
  if constexpr (XT) a_voff = lane * 16;
  else a_voff = ((lane & 15) * ldx + 8 * (lane >> 4)) * 2;
  const int sb = min((n0 >> 6) + (wave >> 1), last_sb);
  const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16_t*>(W + (size_t)sb * KS * 2048), 0, KS * 4096, 0x00020000);

  auto issue_a = [&](int st) {
    bf16_t* so = smem + (st & (kLgStages - 1)) * kLgStageElems;
    if constexpr (GR) {
      const uint32_t dv = XT ? st * 1024u : st * 64u;
#pragma unroll
      for (int i = 0; i < 2; ++i) dma16(ra[0], g_voff[i] + dv, so + (2 * wave + i) * 512);
    } else {
      const uint32_t v = a_voff + (XT ? st * 1024u : st * 64u);
#pragma unroll
      for (int i = 0; i < 2; ++i) dma16(ra[i], v, so + (2 * wave + i) * 512);
    }
  };
  auto issue_b = [&](int st) {
    bf16_t* so = smem + (st & (kLgStages - 1)) * kLgStageElems;
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      const int tt = 2 * (wave & 1) + t2;
      dma16(rb, st * 4096u + tt * 1024u + lane * 16, so + 16 * 512 + ((wave >> 1) * 4 + tt) * 512);
    }
  };
  // wait until stage st has landed.  When it is waited for, stage st + 1 is
  // fully issued and stage st + 2 only its A half (issue_b of a stage follows
  // the barrier), so up to 4 + 2 younger loads may stay outstanding.
  // every iteration issues a full stage (stages past the last one load zeros
  // or unused rows into a buffer nobody reads again), so when stage st is
  // waited for, stage st + 1 is fully issued and st + 2 only its A half
  auto wait_stage = [&](int) { wait_vmcnt<kLgDmaPerStage + kLgDmaPerStage / 2>(); };

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // LDS read offsets (elements, within a stage) of this lane's operand runs.
  // A: m-tile mt covers row blocks wm*8 + 2 mt + {0, 1}; lane rows l % 32.
  // B: n-tile nt is half (nt & 1) of superblock wn*2 + nt/2 (the gate or up
  // half for SwiGLU), fragments 2 (nt & 1) + {0, 1}.
  const int half = (lane >> 4) & 1, r16 = lane & 15, khi = lane >> 5;
  int a_off[4], b_off[2];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) a_off[mt] = (wm * 8 + 2 * mt + half) * 512 + r16 * 8;
#pragma unroll
  for (int nt = 0; nt < 2; ++nt)
    b_off[nt] = 16 * 512 + (wn * 4 + 2 * nt + half) * 512 + r16 * 8;

  struct Frags {
    bf16x8v a[4], b[2];
  };
  // operand runs of 16-k half kk of stage st: run quarter 2 kk + lane / 32
  auto read = [&](Frags& f, int st, int kk) {
    const bf16_t* so = smem + (st & (kLgStages - 1)) * kLgStageElems + (2 * kk + khi) * 128;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) f.a[mt] = *reinterpret_cast<const bf16x8v*>(so + a_off[mt]);
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) f.b[nt] = *reinterpret_cast<const bf16x8v*>(so + b_off[nt]);
  };
  auto mma = [&](const Frags& f) {
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
        acc[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[mt], f.b[nt], acc[mt][nt], 0, 0, 0);
  };

  // Pipeline: up to three stages of direct loads are in flight while one is
  // multiplied.  Iteration kt: the A half of stage kt + 3 (its buffer held
  // stage kt - 1, which every wave finished reading before the last barrier)
  // and the LDS reads of the second half of stage kt are interleaved one per
  // MFMA with the first half's MFMAs; then wait for stage kt + 1, barrier, and
  // interleave the B half of stage kt + 3 and the reads of stage kt + 1's
  // first half with the second half's MFMAs.  sched_group_barrier masks:
  // 0x8 MFMA, 0x100 LDS read, 0x10 vector memory.  Spreading the direct loads
  // this way measured faster than issuing a stage's loads in one burst.
  auto interleave = [&](int nd) {
#pragma unroll
    for (int i = 0; i < 6; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x8, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      if (i < nd) __builtin_amdgcn_sched_group_barrier(0x10, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x8, 2, 0);
  };
  Frags f0, f1;
  for (int st = 0; st < 3; ++st) {
    issue_a(st);
    issue_b(st);
  }
  wait_vmcnt<2 * kLgDmaPerStage>();  // stage 0 landed
  lds_barrier();
  read(f0, 0, 0);
  for (int kt = 0; kt < KS; ++kt) {
    issue_a(kt + 3);
    read(f1, kt, 1);
    mma(f0);
    interleave(2);
    __builtin_amdgcn_sched_barrier(0);
    // (after the last stage this reads a stale buffer that is never used:
    // keeping the step unconditional keeps the LDS reads interleaved)
    wait_stage(kt + 1);
    wait_lgkm0();
    lds_barrier();
    issue_b(kt + 3);
    read(f0, kt + 1, 0);
    mma(f1);
    interleave(2);
    __builtin_amdgcn_sched_barrier(0);
  }
  wait_vmcnt<0>();

  // ---- epilogue.  Accumulator element e of tile (mt, nt): row
  // 8 (e / 4) + 4 (lane / 32) + e % 4, column lane % 32.
  const int col_l = lane & 31;
  auto row_of = [&](int mt, int e) { return m0 + wm * 128 + mt * 32 + 8 * (e >> 2) + 4 * khi + (e & 3); };
  if constexpr (EPI == 2) {
    const int F = N >> 1;
    {
      const int sbg = (n0 >> 6) + wn, j = 0;
      if (sbg <= last_sb) {
      const int f = sbg * 32 + col_l;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = row_of(mt, e);
          if (row < rows) {
            const float gt = acc[mt][2 * j][e], u = acc[mt][2 * j + 1][e];
            const float v = gt / (1.f + __expf(-gt)) * u;
            const size_t off =
                out_tiled ? act_tile_offset(row, f, F) : (size_t)(ent0 + row) * F + f;
            out_bf16[off] = f32_to_bf16(v);
          }
        }
      }
    }
  } else if constexpr (EPI == 3) {
    // grouped down: row = entry ent0 + row of the expert -> (token, slot).
    // The tile's 256 output rows and routing weights are staged in LDS first
    // (read per row in the loop below, the dependent assign -> weight loads
    // were 128 round trips per lane); every wave's direct loads have landed
    // (wait above), so after the barrier the stage buffers are free.
    lds_barrier();
    int* t_row = reinterpret_cast<int*>(smem);
    float* t_wt = reinterpret_cast<float*>(smem) + kLgBM;
    {
      const int row = m0 + threadIdx.x;  // the first 256 threads, one tile row each
      if (threadIdx.x < kLgBM && row < rows) {
        const int asg = g.assign[ent0 + row];
        const int tok = asg / g.k, slot = asg - tok * g.k;
        t_row[threadIdx.x] = slot * g.n + tok;
        t_wt[threadIdx.x] = g.weights[asg];
      }
    }
    lds_barrier();
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = row_of(mt, e);
        if (row >= rows) continue;
        const int lr = row - m0;
        const float wt = t_wt[lr];
        float* dst = out + (size_t)t_row[lr] * ldo;
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          const int col = n0 + wn * 64 + nt * 32 + col_l;
          if (col < N) dst[col] = acc[mt][nt][e] * wt;
        }
      }
  } else {
    // a whole 32-row m-tile inside M takes the unmasked path; for the update
    // form all 64 old values of an n-tile pair are loaded before any store so
    // the loads overlap
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      const bool full = m0 + wm * 128 + mt * 32 + 32 <= M;
#pragma unroll
      for (int np = 0; np < 1; ++np) {
        float old[2][16];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int nt = 2 * np + h;
          const int col = n0 + wn * 64 + nt * 32 + col_l;
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            old[h][e] = 0.f;
            if constexpr (EPI == 1) {
              const int row = row_of(mt, e);
              if ((full || row < M) && col < N) old[h][e] = out[(size_t)row * ldo + col];
            }
          }
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int nt = 2 * np + h;
          const int col = n0 + wn * 64 + nt * 32 + col_l;
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int row = row_of(mt, e);
            if ((full || row < M) && col < N) out[(size_t)row * ldo + col] = old[h][e] + acc[mt][nt][e];
          }
        }
      }
    }
  }
}

bool gemm_large_supported(int m, int n_out, int k) {
  return m >= 1 && n_out % 64 == 0 && k % kLgBK == 0 && k >= kLgBK;
}

hipError_t launch_gemm_large(int m, int n_out, int k, int ldx, int x_tiled, int mode,
                             const bf16_t* x, const bf16_t* w, void* out, int out_tiled,
                             hipStream_t st) {
  if (m == 0) return hipSuccess;
  const int tiles_m = (m + kLgBM - 1) / kLgBM, tiles_n = (n_out + kLgBN - 1) / kLgBN;
  const dim3 grid(tiles_m * tiles_n), block(64 * kLgWaves);
  float* of = reinterpret_cast<float*>(out);
  bf16_t* ob = reinterpret_cast<bf16_t*>(out);
  const GroupArgs none{};
#define SEVO_LG(E, T) \
  hipLaunchKernelGGL((gemm_large_kernel<E, T, 0>), grid, block, 0, st, x, ldx, m, w, n_out, k, of, \
                     n_out, ob, out_tiled, tiles_m, tiles_n, none)
  if (x_tiled) {
    if (mode == 0) SEVO_LG(0, 1);
    else if (mode == 1) SEVO_LG(1, 1);
    else SEVO_LG(2, 1);
  } else {
    if (mode == 0) SEVO_LG(0, 0);
    else if (mode == 1) SEVO_LG(1, 0);
    else SEVO_LG(2, 0);
  }
#undef SEVO_LG
  return hipGetLastError();
}

hipError_t launch_gemm_grouped(int down, int m, int n_out, int k, const bf16_t* x,
                               const bf16_t* w, void* out, const GroupArgs& g, int max_tiles_m,
                               hipStream_t st) {
  if (m == 0 || max_tiles_m == 0) return hipSuccess;
  const int tiles_n = (n_out + kLgBN - 1) / kLgBN;
  const dim3 grid(max_tiles_m * tiles_n), block(64 * kLgWaves);
  if (down)
    hipLaunchKernelGGL((gemm_large_kernel<3, 0, 1>), grid, block, 0, st, x, k, m, w, n_out, k,
                       static_cast<float*>(out), n_out, nullptr, 0, max_tiles_m, tiles_n, g);
  else
    hipLaunchKernelGGL((gemm_large_kernel<2, 1, 1>), grid, block, 0, st, x, k, m, w, n_out, k,
                       nullptr, n_out, static_cast<bf16_t*>(out), 0, max_tiles_m, tiles_n, g);
  return hipGetLastError();
}

}  // namespace sevo
