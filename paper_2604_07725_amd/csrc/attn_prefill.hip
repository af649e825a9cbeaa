// Causal GQA attention of a prefill over the paged KV cache, on the gfx950
// matrix cores.  A prefill (the confidence engine's scoring pass over a whole
// aggregation prompt and trajectory) attends every token of a sequence to all
// keys up to its own position: O(T^2) work, compute-bound, unlike decode.
//
//   * one 256-thread workgroup per (sequence, group of 4 query units, kv
//     head), where a unit is one query head of the kv head's group over 64
//     consecutive tokens; each wave owns one unit;
//   * scores are computed transposed, S^T = K Q^T, with 32x32x16 bf16 MFMAs:
//     a lane then holds one query (lane % 32) and 16 of each 32-key tile's
//     scores, so the online-softmax max and sum are in-lane plus one
//     permlane32 swap; the running max, sum and the output rescale are per
//     lane;
//   * O^T = V^T P^T with the same instruction; P^T's B operand is made from
//     the score accumulators by one permlane32 swap per 8 keys (no LDS);
//   * keys stream in blocks of 64 (4 pages): each wave loads one page (its K
//     and V tiles, 8 KB at head_dim 128) straight into LDS with direct loads
//     through a per-page buffer descriptor -- a page id outside the pool, or a
//     page past the workgroup's keys, gets zero records and reads zeros; three
//     LDS stages keep two blocks of loads in flight;
//   * LDS holds the tiles with their 16-byte chunks XOR-swizzled (within each
//     1 KB) so every MFMA operand read is free of bank conflicts for 8- and
//     16-lane groups; the direct loads apply the swizzle through their
//     per-lane source offsets;
//   * blocks entirely above a wave's queries skip their MFMAs (the wave still
//     loads its page and meets the barriers); workgroups are launched latest
//     (longest) query blocks first.
// P is rounded to bf16 for the P V product (fp32 accumulation); the softmax
// statistics stay fp32.
#include "common.h"
#include "kernels.h"

namespace sevo {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kPfStages = 3;

// K tile block (16 slots x 32 dims, 1 KB): chunk (slot s, dim quarter q) at
// s * 4 + (q ^ pf_kswz(s)).  V tile (dims x 16 slots): chunk (dim e, key half
// h) at e * 2 + (h ^ pf_vswz(e)).
__device__ __forceinline__ int pf_kswz(int s) { return ((s >> 1) ^ (s >> 2)) & 3; }
__device__ __forceinline__ int pf_vswz(int e) { return ((e >> 2) ^ (e >> 3)) & 1; }

template <int D>
__global__ __launch_bounds__(256, 1) void attn_prefill_kernel(PrefillAttnArgs a) {
  constexpr int KT_ELEMS = 16 * D;             // K tile (= V tile) elements
  constexpr int PAGE_ELEMS = 2 * KT_ELEMS;     // (page, head): K tile then V tile
  constexpr int STAGE_ELEMS = 4 * PAGE_ELEMS;  // 4 pages = 64 keys
  constexpr int KB = D / 32;                   // 1 KB blocks per tile
  constexpr int DMA = 2 * KB;                  // direct loads per wave per block
  constexpr int KS = D / 16;                   // 16-dim MFMA steps of q . k
  __shared__ __attribute__((aligned(1024))) bf16_t smem[kPfStages * STAGE_ELEMS];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int sq = blockIdx.z, c = blockIdx.y;
  const int g = a.hq / a.hkv;
  const int seq0 = a.seq_starts[sq];
  const int L = a.seq_starts[sq + 1] - seq0;
  const int p0 = a.start_pos ? a.start_pos[sq] : 0;
  const int units = ((L + 63) >> 6) * g;
  const int ug = gridDim.x - 1 - blockIdx.x;  // latest query blocks first
  if (L <= 0 || 4 * ug >= units) return;      // uniform over the workgroup
  const int u = 4 * ug + wave;
  const bool active = u < units;  // wave-uniform
  const int qb = active ? u / g : 0;
  const int head = c * g + (active ? u % g : 0);
  // keys [0, kend) cover the last query of the workgroup's last unit
  const int qb_last = min(4 * ug + 3, units - 1) / g;
  const int kend = p0 + min(L, 64 * qb_last + 64);
  const int nkb = (kend + 63) >> 6;
  const int npages = (kend + 15) >> 4;
  const int qlo = p0 + 64 * qb;  // position of the wave's first query
  const int last_b = (qlo + 63) >> 6;  // blocks past this hold no key of the wave's rows

  // ---- direct loads: wave w loads page 4 b + w of block b
  // per-lane byte offsets inside a (page, head) region: K block kb chunk lane
  // -> global (slot lane/4, quarter (lane%4) ^ swz); V block vb chunk -> (dim
  // 32 vb + lane/2, half (lane%2) ^ swz)
  const uint32_t k_src = (lane >> 2) * 64 + (((lane & 3) ^ pf_kswz(lane >> 2)) * 16);
  const uint32_t v_src = KT_ELEMS * 2 + (lane >> 1) * 32 + (((lane & 1) ^ pf_vswz(lane >> 1)) * 16);
  auto issue = [&](int b) {
    const int pi = 4 * b + wave;
    int page = -1;
    if (pi < npages && pi < a.max_pages) page = a.page_table[(size_t)sq * a.max_pages + pi];
    const bool ok = page >= 0 && (int64_t)page < a.num_pages;
    const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16_t*>(a.kv_pool + (ok ? ((size_t)page * a.hkv + c) * PAGE_ELEMS : 0)), 0,
        ok ? PAGE_ELEMS * 2 : 0, 0x00020000);
    bf16_t* dst = smem + (b % kPfStages) * STAGE_ELEMS + wave * PAGE_ELEMS;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) dma16(r, k_src + kb * 1024, dst + kb * 512);
#pragma unroll
    for (int vb = 0; vb < KB; ++vb) dma16(r, v_src + vb * 1024, dst + KT_ELEMS + vb * 512);
  };

  // ---- queries of this wave as the B operand of S^T = K Q^T: tile qt holds
  // tokens 32 qt + lane % 32, dims 16 j + 8 (lane / 32) .. + 8 of step j
  const int khi = lane >> 5, l32 = lane & 31;
  bf16x8v qf[2][KS];
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    const int tok = seq0 + min(64 * qb + 32 * qt + l32, L - 1);
    const bf16_t* qp = a.q + ((size_t)tok * a.hq + head) * D + 8 * khi;
#pragma unroll
    for (int j = 0; j < KS; ++j) qf[qt][j] = *reinterpret_cast<const bf16x8v*>(qp + 16 * j);
  }
  int qpos[2];
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) qpos[qt] = qlo + 32 * qt + l32;

  // LDS read offsets (elements) of this lane's operand runs, within a stage.
  // K of key tile kt, step j: key 32 kt + lane % 32 -> page 2 kt + (lane % 32) / 16,
  // slot lane % 16, dim block j / 2, quarter 2 (j % 2) + lane / 32.
  int k_rd[2];
#pragma unroll
  for (int jp = 0; jp < 2; ++jp) {
    const int sl = lane & 15;
    k_rd[jp] = (l32 >> 4) * PAGE_ELEMS + (sl * 4 + ((2 * jp + khi) ^ pf_kswz(sl))) * 8;
  }
  // V of dim tile dt, step j (= page j of the block): dim 32 dt + lane % 32,
  // key half lane / 32
  const int v_rd = KT_ELEMS + (l32 * 2 + (khi ^ pf_vswz(l32))) * 8;

  f32x16 acc_o[KB][2];
#pragma unroll
  for (int dt = 0; dt < KB; ++dt)
#pragma unroll
    for (int qt = 0; qt < 2; ++qt)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc_o[dt][qt][e] = 0.f;
  float m_run[2] = {-INFINITY, -INFINITY}, l_run[2] = {0.f, 0.f};
  const float sl2 = a.scale * 1.4426950408889634f;  // scores in the exp2 domain

  issue(0);
  if (nkb > 1) issue(1);
  if (nkb > 1) wait_vmcnt<DMA>();
  else wait_vmcnt<0>();
  lds_barrier();

  for (int b = 0; b < nkb; ++b) {
    if (b + 2 < nkb) issue(b + 2);  // its buffer held block b - 1, read before the last barrier
    if (active && b <= last_b) {
      const bf16_t* so = smem + (b % kPfStages) * STAGE_ELEMS;
      // ---- S^T for the block: 2 key tiles x 2 query tiles
      f32x16 acc_s[2][2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int qt = 0; qt < 2; ++qt)
#pragma unroll
          for (int e = 0; e < 16; ++e) acc_s[kt][qt][e] = 0.f;
#pragma unroll
      for (int j = 0; j < KS; ++j) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          const bf16x8v kf = *reinterpret_cast<const bf16x8v*>(
              so + 2 * kt * PAGE_ELEMS + (j >> 1) * 512 + k_rd[j & 1]);
#pragma unroll
          for (int qt = 0; qt < 2; ++qt)
            acc_s[kt][qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[qt][j], acc_s[kt][qt], 0, 0, 0);
        }
      }
      // ---- online softmax per query (lane % 32 of each query tile); element
      // e of key tile kt is key 64 b + 32 kt + 8 (e / 4) + 4 (lane / 32) + e % 4
      const bool diag = 64 * b + 63 > qlo;
      bf16x8v pf[2][4];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            float v = acc_s[kt][qt][e] * sl2;
            if (diag) {
              const int key = 64 * b + 32 * kt + 8 * (e >> 2) + 4 * khi + (e & 3);
              if (key > qpos[qt]) v = -INFINITY;
            }
            acc_s[kt][qt][e] = v;
            mx = fmaxf(mx, v);
          }
        mx = xor32_max(mx);
        const float m_new = fmaxf(m_run[qt], mx);  // finite: key 0 is in every row's first block
        const float alpha = exp2f(m_run[qt] - m_new);
        m_run[qt] = m_new;
        float sum = 0.f;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const float p = exp2f(acc_s[kt][qt][e] - m_new);
            acc_s[kt][qt][e] = p;
            sum += p;
          }
        l_run[qt] = l_run[qt] * alpha + xor32_sum(sum);
#pragma unroll
        for (int dt = 0; dt < KB; ++dt) acc_o[dt][qt] *= alpha;
        // B operand of step j (keys 16 j .. 16 j + 15 of the block): lane < 32
        // needs keys +0..7, lane >= 32 keys +8..15.  Lane l holds keys 0-3 and
        // 8-11 of each 16 (lane l + 32 holds 4-7 and 12-15): one swap of the
        // upper half's first group with the lower half's second group.
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int kt = j >> 1, e0 = 8 * (j & 1);
          uint32_t x0 = pack_bf16x2(acc_s[kt][qt][e0 + 0], acc_s[kt][qt][e0 + 1]);
          uint32_t x1 = pack_bf16x2(acc_s[kt][qt][e0 + 2], acc_s[kt][qt][e0 + 3]);
          uint32_t y0 = pack_bf16x2(acc_s[kt][qt][e0 + 4], acc_s[kt][qt][e0 + 5]);
          uint32_t y1 = pack_bf16x2(acc_s[kt][qt][e0 + 6], acc_s[kt][qt][e0 + 7]);
          const auto s0 = __builtin_amdgcn_permlane32_swap(x0, y0, false, false);
          const auto s1 = __builtin_amdgcn_permlane32_swap(x1, y1, false, false);
          const u32x4 w = {s0[0], s1[0], s0[1], s1[1]};
          pf[qt][j] = __builtin_bit_cast(bf16x8v, w);
        }
      }
      // ---- O^T += V^T P^T
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int dt = 0; dt < KB; ++dt) {
          const bf16x8v vf =
              *reinterpret_cast<const bf16x8v*>(so + j * PAGE_ELEMS + dt * 512 + v_rd);
#pragma unroll
          for (int qt = 0; qt < 2; ++qt)
            acc_o[dt][qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[qt][j], acc_o[dt][qt], 0, 0, 0);
        }
    }
    // block b + 1 landed (block b + 2 may stay in flight); every wave is done
    // with block b before anyone refills its buffer
    if (b + 2 < nkb) wait_vmcnt<DMA>();
    else wait_vmcnt<0>();
    wait_lgkm0();
    lds_barrier();
  }

  if (!active) return;
  // ---- out = O / l.  Element e of acc_o[dt][qt]: dim 32 dt + 8 (e / 4) +
  // 4 (lane / 32) + e % 4 of token 32 qt + lane % 32; 4 dims per 8-byte store.
  const int ld = a.hq * D;
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    const int t = 64 * qb + 32 * qt + l32;
    if (t >= L) continue;
    const int row = seq0 + t;
    const float inv = 1.f / l_run[qt];
#pragma unroll
    for (int dt = 0; dt < KB; ++dt)
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int col = head * D + 32 * dt + 8 * e4 + 4 * khi;
        uint2 w;
        w.x = pack_bf16x2(acc_o[dt][qt][4 * e4 + 0] * inv, acc_o[dt][qt][4 * e4 + 1] * inv);
        w.y = pack_bf16x2(acc_o[dt][qt][4 * e4 + 2] * inv, acc_o[dt][qt][4 * e4 + 3] * inv);
        const size_t off = a.out_tiled ? act_tile_offset(row, col, ld) : (size_t)row * ld + col;
        *reinterpret_cast<uint2*>(a.out + off) = w;
      }
  }
}

hipError_t launch_attn_prefill(const PrefillAttnArgs& a, hipStream_t st) {
  if (a.n_seqs == 0 || a.max_seq_len <= 0) return hipSuccess;
  const int g = a.hq / a.hkv;
  const int units = ((a.max_seq_len + 63) / 64) * g;
  const dim3 grid((units + 3) / 4, a.hkv, a.n_seqs);
  if (a.d == 128)
    hipLaunchKernelGGL(attn_prefill_kernel<128>, grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(attn_prefill_kernel<64>, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace sevo
