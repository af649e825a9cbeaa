// Mixture-of-experts FFN of a decode step (Qwen3-MoE layout): router logits,
// the top-k experts of each token with a softmax over the selected logits,
// then SwiGLU experts.  At decode every token of the population routes to k
// experts, so a step touches most experts once: the FFN is a stream of the
// selected experts' weights, each multiplied by the few tokens routed to it.
//
//   * route: one wave per token sums the router GEMM's split-K partials (in
//     split order), takes the k largest logits by repeated wave arg-max
//     (value, then lower expert index) and the softmax over them;
//   * plan: one workgroup counts tokens per expert and lays the (token, slot)
//     assignments out expert-major, tokens in order (ranks from per-expert
//     bit rows: a fixed order, results do not depend on scheduling);
//   * experts: a grouped skinny GEMM over (superblocks, expert): each wave
//     streams 32 or 64 rows of one selected expert's packed weights over the
//     whole K range (no cross-wave reduction), activation rows gathered
//     through the expert's entry list.  Gate/up writes silu(g) * u per entry
//     (bf16, row-major); down writes w * y into partial [slot][token][hidden]
//     (fp32), which the next residual add + RMSNorm sums in slot order.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace sevo {

constexpr int kMoeMaxExperts = 256;
constexpr int kMoeMaxTopK = 16;

// ---- route: logits [S][n][E] (split partials) -> sel [n][k], w [n][k]
__global__ __launch_bounds__(64) void moe_route_kernel(const float* __restrict__ part, int S,
                                                       int n, int E, int k,
                                                       int32_t* __restrict__ sel,
                                                       float* __restrict__ w) {
  const int t = blockIdx.x;
  const int lane = threadIdx.x;
  float v[kMoeMaxExperts / 64];
#pragma unroll
  for (int i = 0; i < kMoeMaxExperts / 64; ++i) {
    const int e = lane + 64 * i;
    float acc = -INFINITY;
    if (e < E) {
      // split order; eight splits' loads issued together
      acc = 0.f;
      for (int s0 = 0; s0 < S; s0 += 8) {
        float p[8];
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (s0 + j < S) p[j] = part[((size_t)(s0 + j) * n + t) * E + e];
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (s0 + j < S) acc += p[j];
      }
    }
    v[i] = acc;
  }
  // k rounds of a wave arg-max over the experts not taken yet (value
  // descending, then lower index); an expert is eligible even when its logit
  // is -inf or NaN, so the k experts are always distinct and valid
  float z[kMoeMaxTopK];
  int id[kMoeMaxTopK];
  uint32_t taken = 0;  // bit i: expert lane + 64 i already selected
#pragma unroll
  for (int r = 0; r < kMoeMaxTopK; ++r) {
    z[r] = -INFINITY;
    id[r] = 0;
    if (r >= k) continue;
    // this lane's best (index ascending with i: strict > keeps the lowest)
    float bv = -INFINITY;
    int bi = 0x7FFFFFFF;
#pragma unroll
    for (int i = 0; i < kMoeMaxExperts / 64; ++i) {
      const int e = lane + 64 * i;
      if (e < E && !((taken >> i) & 1u) && (bi == 0x7FFFFFFF || v[i] > bv)) {
        bv = v[i];
        bi = e;
      }
    }
    // wave arg-max in registers: quads, 8-lane halves of rows and rows by
    // DPP, then pairs of rows and the two halves of the wave by the permlane
    // swaps (each step merges a lane's pair with another lane's; the merge is
    // symmetric, so both lanes keep the same pair)
    auto merge = [&](float ov, int oi) {
      if (oi != 0x7FFFFFFF && (bi == 0x7FFFFFFF || ov > bv || (ov == bv && oi < bi))) {
        bv = ov;
        bi = oi;
      }
    };
    auto dpp_step = [&](auto ctrl) {
      constexpr int C = decltype(ctrl)::value;
      merge(dpp<C>(bv), __builtin_amdgcn_update_dpp(0, bi, C, 0xF, 0xF, false));
    };
    dpp_step(std::integral_constant<int, kDppQuadXor1>{});
    dpp_step(std::integral_constant<int, kDppQuadXor2>{});
    dpp_step(std::integral_constant<int, kDppRowHalfMirror>{});
    dpp_step(std::integral_constant<int, kDppRowMirror>{});
    {
      const auto pv = __builtin_amdgcn_permlane16_swap(__float_as_int(bv), __float_as_int(bv), false, false);
      const auto pi = __builtin_amdgcn_permlane16_swap(bi, bi, false, false);
      bv = __int_as_float(pv[0]);
      bi = pi[0];
      merge(__int_as_float(pv[1]), pi[1]);
    }
    {
      const auto pv = __builtin_amdgcn_permlane32_swap(__float_as_int(bv), __float_as_int(bv), false, false);
      const auto pi = __builtin_amdgcn_permlane32_swap(bi, bi, false, false);
      bv = __int_as_float(pv[0]);
      bi = pi[0];
      merge(__int_as_float(pv[1]), pi[1]);
    }
    // lane 0's choice for every lane (the order is total unless a NaN is
    // involved; then lanes could disagree)
    bi = __builtin_amdgcn_readfirstlane(bi);
    bv = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(bv)));
#pragma unroll
    for (int i = 0; i < kMoeMaxExperts / 64; ++i)
      if (lane + 64 * i == bi) taken |= 1u << i;
    z[r] = bv;
    id[r] = bi;
  }
  if (lane == 0) {
    float sum = 0.f;
#pragma unroll
    for (int r = 0; r < kMoeMaxTopK; ++r)
      if (r < k) sum += expf(z[r] - z[0]);
#pragma unroll
    for (int r = 0; r < kMoeMaxTopK; ++r)
      if (r < k) {
        sel[t * k + r] = id[r];
        w[t * k + r] = expf(z[r] - z[0]) / sum;
      }
  }
}

// ---- plan: offsets [E + 1] and assign [n k] (entries t * k + slot), one
// workgroup.  Counts by LDS atomics; then the entries, 1024 at a time, set
// their bit in a per-expert bit row, and an entry's rank among the entries of
// its expert is the number of set bits before it: the lists are in entry
// (token, slot) order whatever the scheduling.
constexpr int kPlanThreads = 1024;
constexpr int kPlanWords = kPlanThreads / 32;

__global__ __launch_bounds__(kPlanThreads) void moe_plan_kernel(const int32_t* __restrict__ sel,
                                                                int nk, int E,
                                                                int32_t* __restrict__ offsets,
                                                                int32_t* __restrict__ assign,
                                                                int32_t* __restrict__ tile_off) {
  __shared__ int cnt[kMoeMaxExperts];
  __shared__ int base[kMoeMaxExperts];
  __shared__ uint32_t bits[kMoeMaxExperts][kPlanWords];
  const int tid = threadIdx.x;
  for (int e = tid; e < E; e += kPlanThreads) cnt[e] = 0;
  __syncthreads();
  for (int r = tid; r < nk; r += kPlanThreads) {
    const int e = sel[r];
    if (e >= 0 && e < E) atomicAdd(&cnt[e], 1);
  }
  __syncthreads();
  if (tid < 64) {
    // exclusive prefixes over the experts (lane j scans experts 4j..4j+3,
    // E <= 256): entry offsets, and (tile_off) the first 256-entry tile of
    // each expert for the grouped large-M GEMM
    int v[4], tv[4], sum = 0, tsum = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = 4 * tid + u;
      v[u] = e < E ? cnt[e] : 0;
      tv[u] = (v[u] + kMoeGroupRows - 1) / kMoeGroupRows;
      sum += v[u];
      tsum += tv[u];
    }
    int incl = sum, tincl = tsum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(incl, o, kWave);
      const int ty = __shfl_up(tincl, o, kWave);
      if (tid >= o) {
        incl += y;
        tincl += ty;
      }
    }
    int run = incl - sum, trun = tincl - tsum;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = 4 * tid + u;
      if (e < E) {
        base[e] = run;
        offsets[e] = run;
        if (tile_off) tile_off[e] = trun;
      }
      run += v[u];
      trun += tv[u];
    }
    if (tid == 63) {
      offsets[E] = incl;
      if (tile_off) tile_off[E] = tincl;
    }
  }
  for (int c0 = 0; c0 < nk; c0 += kPlanThreads) {
    for (int w = tid; w < E * kPlanWords; w += kPlanThreads) (&bits[0][0])[w] = 0u;
    __syncthreads();  // orders the prefix (first chunk) before the reads of base
    const int r = c0 + tid;
    const int e = r < nk ? sel[r] : -1;
    const bool ok = e >= 0 && e < E;
    if (ok) atomicOr(&bits[e][tid >> 5], 1u << (tid & 31));
    __syncthreads();
    if (ok) {
      int rank = __popc(bits[e][tid >> 5] & ((1u << (tid & 31)) - 1u));
      for (int w = 0; w < (tid >> 5); ++w) rank += __popc(bits[e][w]);
      assign[base[e] + rank] = r;
    }
    __syncthreads();
    for (int x = tid; x < E; x += kPlanThreads) {
      int tot = 0;
      for (int w = 0; w < kPlanWords; ++w) tot += __popc(bits[x][w]);
      base[x] += tot;
    }
    __syncthreads();  // the bit rows are read above before the next chunk clears them
  }
}

// ---- the same plan for many entries (a prefill chunk), in three launches
// that give identical offsets, tiles and lists: (1) a workgroup per 1024-entry
// chunk counts its entries per expert; (2) one workgroup turns the counts into
// each (chunk, expert)'s first list position, plus offsets and tile_off;
// (3) a workgroup per chunk ranks its entries by the same bit rows as above.
__global__ __launch_bounds__(kPlanThreads) void moe_plan_count_kernel(
    const int32_t* __restrict__ sel, int nk, int E, int32_t* __restrict__ ccnt) {
  __shared__ int cnt[kMoeMaxExperts];
  const int tid = threadIdx.x;
  for (int e = tid; e < E; e += kPlanThreads) cnt[e] = 0;
  __syncthreads();
  const int r = blockIdx.x * kPlanThreads + tid;
  if (r < nk) {
    const int e = sel[r];
    if (e >= 0 && e < E) atomicAdd(&cnt[e], 1);
  }
  __syncthreads();
  for (int e = tid; e < E; e += kPlanThreads) ccnt[(size_t)blockIdx.x * E + e] = cnt[e];
}

// ccnt [chunks][E] counts in, first positions out.  Thread (part p, expert e)
// walks a quarter of the chunks (E <= 256).
__global__ __launch_bounds__(kPlanThreads) void moe_plan_scan_kernel(
    int32_t* __restrict__ ccnt, int chunks, int E, int32_t* __restrict__ offsets,
    int32_t* __restrict__ tile_off) {
  constexpr int kParts = kPlanThreads / kMoeMaxExperts;
  __shared__ int psum[kParts][kMoeMaxExperts];
  __shared__ int ebase[kMoeMaxExperts];
  const int tid = threadIdx.x;
  const int p = tid / kMoeMaxExperts, e = tid % kMoeMaxExperts;
  const int per = (chunks + kParts - 1) / kParts;
  const int c0 = min(chunks, p * per), c1 = min(chunks, c0 + per);
  int sum = 0;
  if (e < E)
    for (int c = c0; c < c1; ++c) sum += ccnt[(size_t)c * E + e];
  psum[p][e] = sum;
  __syncthreads();
  if (tid < 64) {
    // exclusive prefixes over the experts (lane j: experts 4j..4j+3): entry
    // offsets and the first 256-entry tile of each expert
    int v[4], tv[4], tot = 0, ttot = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int x = 4 * tid + u;
      v[u] = 0;
      if (x < E)
#pragma unroll
        for (int q = 0; q < kParts; ++q) v[u] += psum[q][x];
      tv[u] = (v[u] + kMoeGroupRows - 1) / kMoeGroupRows;
      tot += v[u];
      ttot += tv[u];
    }
    int incl = tot, tincl = ttot;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(incl, o, kWave);
      const int ty = __shfl_up(tincl, o, kWave);
      if (tid >= o) {
        incl += y;
        tincl += ty;
      }
    }
    int run = incl - tot, trun = tincl - ttot;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int x = 4 * tid + u;
      if (x < E) {
        ebase[x] = run;
        offsets[x] = run;
        if (tile_off) tile_off[x] = trun;
      }
      run += v[u];
      trun += tv[u];
    }
    if (tid == 63) {
      offsets[E] = incl;
      if (tile_off) tile_off[E] = tincl;
    }
  }
  __syncthreads();
  if (e < E) {
    int run = ebase[e];
    for (int q = 0; q < p; ++q) run += psum[q][e];
    for (int c = c0; c < c1; ++c) {
      const int v = ccnt[(size_t)c * E + e];
      ccnt[(size_t)c * E + e] = run;
      run += v;
    }
  }
}

__global__ __launch_bounds__(kPlanThreads) void moe_plan_place_kernel(
    const int32_t* __restrict__ sel, int nk, int E, const int32_t* __restrict__ cbase,
    int32_t* __restrict__ assign) {
  __shared__ uint32_t bits[kMoeMaxExperts][kPlanWords];
  const int tid = threadIdx.x;
  for (int w = tid; w < E * kPlanWords; w += kPlanThreads) (&bits[0][0])[w] = 0u;
  __syncthreads();
  const int r = blockIdx.x * kPlanThreads + tid;
  const int e = r < nk ? sel[r] : -1;
  const bool ok = e >= 0 && e < E;
  if (ok) atomicOr(&bits[e][tid >> 5], 1u << (tid & 31));
  __syncthreads();
  if (ok) {
    int rank = __popc(bits[e][tid >> 5] & ((1u << (tid & 31)) - 1u));
    for (int w = 0; w < (tid >> 5); ++w) rank += __popc(bits[e][w]);
    assign[cbase[(size_t)blockIdx.x * E + e] + rank] = r;
  }
}

size_t moe_plan_scratch_bytes(int nk, int E) {
  return (size_t)((nk + kPlanThreads - 1) / kPlanThreads) * E * 4;
}

// Grouped skinny GEMM over the selected experts.  At decode an expert sees a
// few tokens, so the kernel is a stream of the selected experts' weights.
// A wave takes FPW of the four 16-row fragments of one 64-row weight
// superblock over the whole K range, so no partial sum crosses waves (no LDS,
// no barrier); a workgroup's four waves take 4 FPW / 4 superblocks:
//   EPI 0 (gate/up): gate fragment f pairs with up fragment f + 2 (the 32 + 32
//     superblock), SwiGLU in registers; X = the normed input, tiled [n][H],
//     rows gathered by token; out act [n k][Fe] bf16, row = entry position;
//   EPI 1 (down): X = the expert's act rows; out part [k][n][H] fp32 =
//     routing weight * product.
// FPW is chosen so the grid fits one round of resident waves.  The expert's
// entries come in tiles of 16 NB rows (NB from the expected entries per
// expert); an expert with more entries takes further tiles, re-reading its
// weights.  Four fragment buffers keep three steps' loads in flight.
template <int NB, int FPW>
struct MoeFrag {
  bf16x8v a[FPW];
  bf16x8v b[NB];
};

template <int EPI, int NB, int FPW>
__global__ __launch_bounds__(256) void moe_expert_kernel(MoeExpertArgs a) {
  static_assert(FPW == 2 || FPW == 4, "two or four fragments per wave");
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int e = blockIdx.y;
  const int off = a.offsets[e];
  const int ne = a.offsets[e + 1] - off;
  const int K = EPI == 0 ? a.hidden : a.ffn;
  const int N = EPI == 0 ? 2 * a.ffn : a.hidden;
  constexpr int kSbPerGroup = FPW;  // superblocks per workgroup (4 waves)
  const int sb = kSbPerGroup * blockIdx.x + wave / (4 / FPW);
  if (ne <= 0 || sb >= N / 64) return;  // wave-uniform; no barrier follows
  const int KS = K >> 5;
  const int p = wave & 1;  // which half of the superblock (FPW = 2)
  // the wave's fragments; for gate/up, pairs (gate, up) are adjacent
  int fr[FPW];
  if constexpr (FPW == 4) {
    if constexpr (EPI == 0) { fr[0] = 0; fr[1] = 2; fr[2] = 1; fr[3] = 3; }
    else { fr[0] = 0; fr[1] = 1; fr[2] = 2; fr[3] = 3; }
  } else {
    if constexpr (EPI == 0) { fr[0] = p; fr[1] = p + 2; }
    else { fr[0] = 2 * p; fr[1] = 2 * p + 1; }
  }
  const int r = lane & 15, q = lane >> 4;
  const bf16_t* wp = (EPI == 0 ? a.w_gate_up : a.w_down) + (size_t)e * N * K +
                     (size_t)sb * KS * 2048 + lane * 8;

  for (int m0 = 0; m0 < ne; m0 += 16 * NB) {
    // activation rows of this lane per 16-row block (rows past the expert's
    // count read its last row: they only feed outputs that are never stored)
    const bf16_t* xp[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int i = min(m0 + 16 * b + r, ne - 1);
      if constexpr (EPI == 0) {
        const int t = a.assign[off + i] / a.top_k;
        xp[b] = a.x + ((size_t)(t >> 4) * KS) * 512 + (16 * q + (t & 15)) * 8;
      } else {
        xp[b] = a.act + (size_t)(off + i) * a.ffn + 8 * q;
      }
    }
    f32x4 acc[FPW][NB];
#pragma unroll
    for (int h = 0; h < FPW; ++h)
#pragma unroll
      for (int b = 0; b < NB; ++b) acc[h][b] = f32x4{0.f, 0.f, 0.f, 0.f};
    // step j of K; past the end it re-reads the last one (cache hits, unused).
    // Expert weights are read once: non-temporal loads keep their stream from
    // evicting the gathered activation rows from L2 (experts 211 -> 200 us
    // per layer at the 30B-A3B shape)
    auto load = [&](MoeFrag<NB, FPW>& f, int j) {
      const int st = min(j, KS - 1);
#pragma unroll
      for (int h = 0; h < FPW; ++h)
        f.a[h] = __builtin_nontemporal_load(
            reinterpret_cast<const bf16x8v*>(wp + (size_t)st * 2048 + fr[h] * 512));
#pragma unroll
      for (int b = 0; b < NB; ++b)
        f.b[b] = *reinterpret_cast<const bf16x8v*>(
            xp[b] + (EPI == 0 ? (size_t)st * 512 : (size_t)st * 32));
    };
    auto mma = [&](const MoeFrag<NB, FPW>& f) {
#pragma unroll
      for (int h = 0; h < FPW; ++h)
#pragma unroll
        for (int b = 0; b < NB; ++b)
          acc[h][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.a[h], f.b[b], acc[h][b], 0, 0, 0);
    };
    {
      MoeFrag<NB, FPW> f0, f1, f2, f3;
      load(f0, 0);
      load(f1, 1);
      load(f2, 2);
      for (int j = 0; j < KS; j += 4) {
        load(f3, j + 3);
        __builtin_amdgcn_sched_barrier(0);
        mma(f0);
        __builtin_amdgcn_sched_barrier(0);
        load(f0, j + 4);
        __builtin_amdgcn_sched_barrier(0);
        if (j + 1 < KS) mma(f1);
        __builtin_amdgcn_sched_barrier(0);
        load(f1, j + 5);
        __builtin_amdgcn_sched_barrier(0);
        if (j + 2 < KS) mma(f2);
        __builtin_amdgcn_sched_barrier(0);
        load(f2, j + 6);
        __builtin_amdgcn_sched_barrier(0);
        if (j + 3 < KS) mma(f3);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // D of fragment h, token block b: lane holds entry row 16 b + lane % 16
    // and weight rows 4 (lane / 16) + 0..3 of the fragment (4 consecutive
    // output columns)
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int i = m0 + 16 * b + r;
      if (i >= ne) continue;
      if constexpr (EPI == 0) {
#pragma unroll
        for (int h = 0; h < FPW; h += 2) {
          const f32x4 g = acc[h][b], u = acc[h + 1][b];
          const int col = sb * 32 + 16 * fr[h] + 4 * q;
          uint2 o;
          o.x = pack_bf16x2(g.x / (1.f + __expf(-g.x)) * u.x, g.y / (1.f + __expf(-g.y)) * u.y);
          o.y = pack_bf16x2(g.z / (1.f + __expf(-g.z)) * u.z, g.w / (1.f + __expf(-g.w)) * u.w);
          *reinterpret_cast<uint2*>(a.act + (size_t)(off + i) * a.ffn + col) = o;
        }
      } else {
        const int asg = a.assign[off + i];
        const int t = asg / a.top_k, slot = asg - t * a.top_k;
        const float wt = a.weights[asg];
        float* dst = a.part + ((size_t)slot * a.n + t) * a.hidden + sb * 64 + 4 * q;
#pragma unroll
        for (int h = 0; h < FPW; ++h)
          *reinterpret_cast<f32x4*>(dst + 16 * fr[h]) = acc[h][b] * wt;
      }
    }
  }
}

// Sum of the k slot partials of each row, in slot order: out [n][H] (row
// stride ldo) = sum over j of part [j][n][H].  The prefill's chunks write
// their rows of the residual update this way.
__global__ __launch_bounds__(256) void moe_sum_slots_kernel(const float* __restrict__ part,
                                                            int k, int n, int H,
                                                            float* __restrict__ out) {
  const size_t total4 = (size_t)n * H / 4;
  const size_t plane = (size_t)n * H;
  for (size_t g = (size_t)blockIdx.x * blockDim.x + threadIdx.x; g < total4;
       g += (size_t)gridDim.x * blockDim.x) {
    f32x4 acc = *reinterpret_cast<const f32x4*>(part + g * 4);
    for (int j0 = 1; j0 < k; j0 += 8) {  // slot order; eight slots' loads together
      f32x4 p[8];
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (j0 + j < k) p[j] = *reinterpret_cast<const f32x4*>(part + (j0 + j) * plane + g * 4);
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (j0 + j < k) acc += p[j];
    }
    *reinterpret_cast<f32x4*>(out + g * 4) = acc;
  }
}

hipError_t launch_moe_sum_slots(const float* part, int k, int n, int H, float* out,
                                hipStream_t st) {
  if (n == 0) return hipSuccess;
  const size_t total4 = (size_t)n * H / 4;
  const int grid = (int)std::min<size_t>((total4 + 255) / 256, 4096);
  hipLaunchKernelGGL(moe_sum_slots_kernel, dim3(grid), dim3(256), 0, st, part, k, n, H, out);
  return hipGetLastError();
}

bool moe_supported(int E, int top_k, int ffn, int hidden) {
  return E >= 64 && E <= kMoeMaxExperts && E % 64 == 0 && top_k >= 1 && top_k <= kMoeMaxTopK &&
         top_k <= E && ffn >= 32 && ffn % 32 == 0 && hidden % 64 == 0;
}

hipError_t launch_moe_route(const float* part, int S, int n, int E, int k, int32_t* sel,
                            float* w, hipStream_t st) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(moe_route_kernel, dim3(n), dim3(64), 0, st, part, S, n, E, k, sel, w);
  return hipGetLastError();
}

hipError_t launch_moe_plan(const int32_t* sel, int nk, int E, int32_t* offsets, int32_t* assign,
                           hipStream_t st, int32_t* tile_off, int32_t* scratch) {
  if (scratch && nk > 4 * kPlanThreads) {
    const int chunks = (nk + kPlanThreads - 1) / kPlanThreads;
    hipLaunchKernelGGL(moe_plan_count_kernel, dim3(chunks), dim3(kPlanThreads), 0, st, sel, nk, E,
                       scratch);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
    hipLaunchKernelGGL(moe_plan_scan_kernel, dim3(1), dim3(kPlanThreads), 0, st, scratch, chunks,
                       E, offsets, tile_off);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
    hipLaunchKernelGGL(moe_plan_place_kernel, dim3(chunks), dim3(kPlanThreads), 0, st, sel, nk, E,
                       scratch, assign);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(moe_plan_kernel, dim3(1), dim3(kPlanThreads), 0, st, sel, nk, E, offsets,
                     assign, tile_off);
  return hipGetLastError();
}

hipError_t launch_moe_experts(const MoeExpertArgs& a, hipStream_t st) {
  if (a.n == 0) return hipSuccess;
  // token tile from the expected entries per expert (n k / E): one 16-row
  // block at decode sizes, up to four for prefill-like batches
  const long long per = ((long long)a.n * a.top_k + a.n_experts - 1) / a.n_experts;
  const int nb = per <= 12 ? 1 : (per <= 24 ? 2 : 4);
  // gate/up: 2 fragments per wave (2 superblocks per workgroup); down: the
  // whole superblock per wave (4 per workgroup), so that at the 30B-A3B shape
  // each grid is one round of resident waves
  const dim3 g0((2 * a.ffn / 64 + 1) / 2, a.n_experts), g1((a.hidden / 64 + 3) / 4, a.n_experts);
#define SEVO_MOE_LAUNCH(NB)                                                          \
  hipLaunchKernelGGL((moe_expert_kernel<0, NB, 2>), g0, dim3(256), 0, st, a);      \
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;                 \
  hipLaunchKernelGGL((moe_expert_kernel<1, NB, 4>), g1, dim3(256), 0, st, a);
  if (nb == 1) {
    SEVO_MOE_LAUNCH(1)
  } else if (nb == 2) {
    SEVO_MOE_LAUNCH(2)
  } else {
    SEVO_MOE_LAUNCH(4)
  }
#undef SEVO_MOE_LAUNCH
  return hipGetLastError();
}

}  // namespace sevo
