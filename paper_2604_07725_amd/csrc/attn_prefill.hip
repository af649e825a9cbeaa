// Causal GQA attention of a prefill over the paged KV cache, on the gfx950
// matrix cores.  A prefill (the confidence engine's scoring pass over a whole
// aggregation prompt and trajectory) attends every token of a sequence to all
// keys up to its own position: O(T^2) work, compute-bound, unlike decode.
//
//   * one workgroup of NW waves per (sequence, NW query units, kv head); a
//     unit is one query head of the kv head's group over 32 NQT consecutive
//     tokens, and each wave owns one unit.  The shipped shape is 12 waves of
//     32 queries: 162 registers per wave, so three waves share each SIMD and
//     the MFMAs of one overlap the softmax of the others (8 waves, two per
//     SIMD, measured 5% slower; 16 waves spill; 4 waves of 64 queries, one per
//     SIMD, 16% slower than 8, and a hand-pipelined single wave spilled);
//   * scores are computed transposed, S^T = K Q^T, with 32x32x16 bf16 MFMAs:
//     a lane then holds one query (lane % 32) and 16 of each 32-key tile's
//     scores, so the online-softmax max and sum are in-lane plus one
//     permlane32 swap; the running max, sum and the output rescale are per
//     lane.  The exp argument is one FMA; the running max is raised (and O
//     rescaled) only when a row's block max exceeds it by more than 8 (a
//     factor 256, harmless in fp32 and bf16);
//   * O^T = V^T P^T with the same instruction; P^T's B operand is made from
//     the score accumulators by one permlane32 swap per 8 keys (no LDS);
//   * keys stream in blocks of 64 (4 pages) straight into LDS with direct
//     loads through a per-page buffer descriptor (waves 0-7, two per page: one
//     K tile, one V tile) -- a page id outside the pool, or a page past the
//     workgroup's keys, gets zero records and reads zeros; four LDS stages
//     hold the block being multiplied and up to three more in flight;
//   * the keys of a page whose id lies outside the pool are left out, as in
//     decode.  Such ids are a caller's error, so the hot loop stays as it is
//     unless the workgroup finds one among its pages in a pre-pass; then each
//     wave learns a block's absent pages when it issues the block (scalar
//     loads of its four page ids, kept as 4 bits per stage) and sets their
//     scores to kAbsentKey, a finite value so far below any real score that
//     its weight is exactly 0 once a real key is seen (a row that sees none
//     gets o = 0, its values being 0);
//   * LDS holds the tiles with their 16-byte chunks XOR-swizzled (within each
//     1 KB) so every MFMA operand read is free of bank conflicts for 8- and
//     16-lane groups; the direct loads apply the swizzle through their
//     per-lane source offsets;
//   * blocks entirely above a wave's queries skip their MFMAs (the wave still
//     loads its part of the block and meets the barriers); workgroups are
//     launched latest (longest) query blocks first, the kv head varying
//     fastest so each head stays on the same XCDs;
//   * the slots of a sequence's last page past its last key may hold anything
//     (NaN included): in the block holding that key they are zeroed in the V
//     tiles (the scores there are masked; K needs nothing).
// P is rounded to bf16 for the P V product (fp32 accumulation); the softmax
// statistics stay fp32.  The exponentials are the bare hardware exp2 (results
// below 2^-126 flush to zero; a row's running max keeps its sum >= 2^-8).
#include "common.h"
#include "kernels.h"

namespace sevo {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kPfStages = 4;
constexpr int kPfWaves = 12;     // waves per workgroup
constexpr int kPfQueryTiles = 1; // 32-query tiles per wave
// Score given to a key on a page outside the pool.  Far below any real score
// (|q . k| of ordinary bf16 inputs is many orders smaller), yet small enough
// that its product with the scale, rounded to fp32, is off by well under 1 in
// the exp2 argument fma(s, scale log2 e, -max): a row that has seen only such
// keys gets weights near 1 on zero values (o = 0), never exp2(+huge) = inf
// (-1e30 would leave an error of ~1e21 there).
constexpr float kAbsentKey = -1e6f;

// K tile block (16 slots x 32 dims, 1 KB): chunk (slot s, dim quarter q) at
// s * 4 + (q ^ pf_kswz(s)).  V tile (dims x 16 slots): chunk (dim e, key half
// h) at e * 2 + (h ^ pf_vswz(e)).
__device__ __forceinline__ int pf_kswz(int s) { return ((s >> 1) ^ (s >> 2)) & 3; }
__device__ __forceinline__ int pf_vswz(int e) { return ((e >> 2) ^ (e >> 3)) & 1; }

template <int D, int NW, int NQT>
__global__ __launch_bounds__(64 * NW, 1) void attn_prefill_kernel(PrefillAttnArgs a) {
  constexpr int KT_ELEMS = 16 * D, PAGE_ELEMS = 2 * KT_ELEMS, STAGE_ELEMS = 4 * PAGE_ELEMS;
  constexpr int KB = D / 32, KS = D / 16, UQ = 32 * NQT;
  constexpr int DMA = NW == 4 ? 2 * KB : KB;
  __shared__ __attribute__((aligned(1024))) bf16_t smem[kPfStages * STAGE_ELEMS];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // the kv head is the fastest-varying part of the launch order, so the
  // round-robin placement of workgroups on the 8 XCDs keeps a head's keys and
  // values in the L2 of the same XCD(s); query groups go latest first
  const int sq = blockIdx.z;
  const int lin = blockIdx.x + gridDim.x * blockIdx.y;  // gridDim.y == hkv
  const int c = lin % a.hkv;
  const int g = a.hq / a.hkv;
  const int seq0 = a.seq_starts[sq];
  const int L = a.seq_starts[sq + 1] - seq0;
  const int p0 = a.start_pos ? a.start_pos[sq] : 0;
  const int units = ((L + UQ - 1) / UQ) * g;
  const int ug = gridDim.x - 1 - lin / a.hkv;
  if (L <= 0 || NW * ug >= units) return;
  const int u = NW * ug + wave;
  const bool active = u < units;
  const int qb = active ? u / g : 0;
  const int head = c * g + (active ? u % g : 0);
  const int qb_last = min(NW * ug + NW - 1, units - 1) / g;
  const int kend = p0 + min(L, UQ * qb_last + UQ);
  const int nkb = (kend + 63) >> 6;
  const int npages = (kend + 15) >> 4;
  const int qlo = p0 + UQ * qb;
  const int last_b = (qlo + UQ - 1) >> 6;

  // ---- direct loads of block b: page 4 b + w (NW = 4: both tiles) or page
  // 4 b + w / 2 (NW = 8: the K tile for even waves, the V tile for odd).
  // Per-lane byte offsets inside a (page, head) region: K block kb chunk lane
  // -> global (slot lane/4, quarter (lane%4) ^ swz); V block vb chunk -> (dim
  // 32 vb + lane/2, half (lane%2) ^ swz)
  const uint32_t k_src = (lane >> 2) * 64 + (((lane & 3) ^ pf_kswz(lane >> 2)) * 16);
  const uint32_t v_src = KT_ELEMS * 2 + (lane >> 1) * 32 + (((lane & 1) ^ pf_vswz(lane >> 1)) * 16);
  // any page of the workgroup's key range outside the pool?  (workgroup-uniform)
  int any_absent = 0;
  for (int p = threadIdx.x; p < npages; p += 64 * NW) {
    const int pg = p < a.max_pages ? a.page_table[(size_t)sq * a.max_pages + p] : -1;
    any_absent |= pg < 0 || (int64_t)pg >= a.num_pages;
  }
  any_absent = __syncthreads_or(any_absent);
  uint32_t absent = 0;  // bit 4 (b % kPfStages) + j: page j of that stage's block is absent
  // the sequence's page ids through the constant address space: the kernel
  // never writes the table, and wave-uniform reads then become scalar loads
  // (a vector load here would make the compiler wait for every outstanding
  // direct load before its result is used)
  const __attribute__((address_space(4))) int32_t* ptab =
      (const __attribute__((address_space(4))) int32_t*)(a.page_table + (size_t)sq * a.max_pages);
  auto issue = [&](int b) {
    const int pi = 4 * b + (NW == 4 ? wave : wave >> 1);
    int page = -1;
    if (pi < npages && pi < a.max_pages) page = ptab[pi];
    if (any_absent) {
      uint32_t bad = 0;
      for (int j = 0; j < 4; ++j) {
        const int pj = 4 * b + j;
        if (pj >= npages) continue;  // past the workgroup's keys: causally masked
        const int pg = pj < a.max_pages ? ptab[pj] : -1;
        if (pg < 0 || (int64_t)pg >= a.num_pages) bad |= 1u << j;
      }
      const int sh = 4 * (b % kPfStages);
      absent = (absent & ~(0xFu << sh)) | (bad << sh);
    }
    const bool ok = page >= 0 && (int64_t)page < a.num_pages;
    const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16_t*>(a.kv_pool + (ok ? ((size_t)page * a.hkv + c) * PAGE_ELEMS : 0)), 0,
        ok ? PAGE_ELEMS * 2 : 0, 0x00020000);
    bf16_t* dst = smem + (b % kPfStages) * STAGE_ELEMS + (NW == 4 ? wave : wave >> 1) * PAGE_ELEMS;
    if (NW > 8 && wave >= 8) return;  // waves 8.. load nothing
    if (NW == 4 || (wave & 1) == 0) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) dma16(r, k_src + kb * 1024, dst + kb * 512);
    }
    if (NW == 4 || (wave & 1) == 1) {
#pragma unroll
      for (int vb = 0; vb < KB; ++vb) dma16(r, v_src + vb * 1024, dst + KT_ELEMS + vb * 512);
    }
  };
  const int khi = lane >> 5, l32 = lane & 31;
  bf16x8v qf[NQT][KS];
  int qpos[NQT];
#pragma unroll
  for (int qt = 0; qt < NQT; ++qt) {
    const int tok = seq0 + min(UQ * qb + 32 * qt + l32, L - 1);
    const bf16_t* qp = a.q + ((size_t)tok * a.hq + head) * D + 8 * khi;
#pragma unroll
    for (int j = 0; j < KS; ++j) qf[qt][j] = *reinterpret_cast<const bf16x8v*>(qp + 16 * j);
    qpos[qt] = qlo + 32 * qt + l32;
  }
  int k_rd[2];
#pragma unroll
  for (int jp = 0; jp < 2; ++jp) {
    const int sl = lane & 15;
    k_rd[jp] = (l32 >> 4) * PAGE_ELEMS + (sl * 4 + ((2 * jp + khi) ^ pf_kswz(sl))) * 8;
  }
  const int v_rd = KT_ELEMS + (l32 * 2 + (khi ^ pf_vswz(l32))) * 8;
  f32x16 acc_o[KB][NQT];
#pragma unroll
  for (int dt = 0; dt < KB; ++dt)
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc_o[dt][qt][e] = 0.f;
  float m_run[NQT], l_run[NQT];
#pragma unroll
  for (int qt = 0; qt < NQT; ++qt) { m_run[qt] = -INFINITY; l_run[qt] = 0.f; }
  const float sl2 = a.scale * 1.4426950408889634f;

  for (int st = 0; st < 3 && st < nkb; ++st) issue(st);
  if (nkb >= 3) wait_vmcnt<2 * DMA>();
  else if (nkb == 2) wait_vmcnt<DMA>();
  else wait_vmcnt<0>();
  lds_barrier();
  const int nkeys = p0 + L;  // the sequence's keys; later slots may hold anything
  // everything issued so far has landed before the first block (the q
  // fragments and the first stages): otherwise the compiler, unable to tell
  // which of those loads are still pending inside the loop, drains the
  // direct loads of later stages at each block's first q use.  Once per
  // workgroup; 1120 -> 1132 TFLOP/s at 40K tokens, with the scalar page ids
  wait_vmcnt<0>();
  for (int b = 0; b < nkb; ++b) {
    if (64 * b + 64 > nkeys) {
      // the block with the sequence's last key: its V slots past that key
      // are zeroed in LDS (P is 0 there, but 0 x NaN would not be); uniform
      // over the workgroup
      bf16_t* so = smem + (b % kPfStages) * STAGE_ELEMS + KT_ELEMS;
      for (int idx = threadIdx.x; idx < 4 * D; idx += 64 * NW) {
        const int j = idx / D, e = idx - (idx / D) * D;
        for (int sl = 0; sl < kPage; ++sl)
          if (64 * b + 16 * j + sl >= nkeys)
            so[j * PAGE_ELEMS + (e * 2 + ((sl >> 3) ^ pf_vswz(e))) * 8 + (sl & 7)] = 0;
      }
      lds_barrier();
    }
    if (active && b <= last_b) {
      const bf16_t* so = smem + (b % kPfStages) * STAGE_ELEMS;
      f32x16 acc_s[2][NQT];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt)
#pragma unroll
          for (int e = 0; e < 16; ++e) acc_s[kt][qt][e] = 0.f;
#pragma unroll
      for (int j = 0; j < KS; ++j)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          const bf16x8v kf = *reinterpret_cast<const bf16x8v*>(so + 2 * kt * PAGE_ELEMS + (j >> 1) * 512 + k_rd[j & 1]);
#pragma unroll
          for (int qt = 0; qt < NQT; ++qt)
            acc_s[kt][qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[qt][j], acc_s[kt][qt], 0, 0, 0);
        }
      const bool diag = 64 * b + 63 > qlo;
      bf16x8v pf[NQT][4];
#pragma unroll
      for (int qt = 0; qt < NQT; ++qt) {
        if (diag) {
#pragma unroll
          for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              const int key = 64 * b + 32 * kt + 8 * (e >> 2) + 4 * khi + (e & 3);
              if (key > qpos[qt]) acc_s[kt][qt][e] = -INFINITY;
            }
        }
        const uint32_t bad = any_absent ? (absent >> (4 * (b % kPfStages))) & 0xFu : 0u;
        if (bad) {
          // element e of tile kt holds a key of page 2 kt + e / 8 of the block
#pragma unroll
          for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int e = 0; e < 16; ++e)
              if ((bad >> (2 * kt + (e >> 3))) & 1u)
                acc_s[kt][qt][e] = fminf(acc_s[kt][qt][e], kAbsentKey);
        }
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int e = 0; e < 16; e += 2) mx = fmaxf(mx, fmaxf(acc_s[kt][qt][e], acc_s[kt][qt][e + 1]));
        mx = xor32_max(mx) * sl2;
        if (__any(mx > m_run[qt] + 8.f)) {
          const float m_new = fmaxf(m_run[qt], mx);
          const float alpha = __builtin_amdgcn_exp2f(m_run[qt] - m_new);
          m_run[qt] = m_new;
          l_run[qt] *= alpha;
#pragma unroll
          for (int dt = 0; dt < KB; ++dt) acc_o[dt][qt] *= alpha;
        }
        const float nm = -m_run[qt];
        float sum = 0.f;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(acc_s[kt][qt][e], sl2, nm));
            acc_s[kt][qt][e] = p;
            sum += p;
          }
        l_run[qt] += xor32_sum(sum);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int kt = j >> 1, e0 = 8 * (j & 1);
          const uint32_t x0 = pack_bf16x2(acc_s[kt][qt][e0 + 0], acc_s[kt][qt][e0 + 1]);
          const uint32_t x1 = pack_bf16x2(acc_s[kt][qt][e0 + 2], acc_s[kt][qt][e0 + 3]);
          const uint32_t y0 = pack_bf16x2(acc_s[kt][qt][e0 + 4], acc_s[kt][qt][e0 + 5]);
          const uint32_t y1 = pack_bf16x2(acc_s[kt][qt][e0 + 6], acc_s[kt][qt][e0 + 7]);
          const auto s0 = __builtin_amdgcn_permlane32_swap(x0, y0, false, false);
          const auto s1 = __builtin_amdgcn_permlane32_swap(x1, y1, false, false);
          const u32x4 w = {s0[0], s1[0], s0[1], s1[1]};
          pf[qt][j] = __builtin_bit_cast(bf16x8v, w);
        }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int dt = 0; dt < KB; ++dt) {
          const bf16x8v vf = *reinterpret_cast<const bf16x8v*>(so + j * PAGE_ELEMS + dt * 512 + v_rd);
#pragma unroll
          for (int qt = 0; qt < NQT; ++qt)
            acc_o[dt][qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[qt][j], acc_o[dt][qt], 0, 0, 0);
        }
    }
    if (b + 1 < nkb) {
      if (b + 2 < nkb) wait_vmcnt<DMA>();
      else wait_vmcnt<0>();
      wait_lgkm0();
      lds_barrier();
      if (b + 3 < nkb) issue(b + 3);
    }
  }
  wait_vmcnt<0>();
  if (!active) return;
  const int ld = a.hq * D;
#pragma unroll
  for (int qt = 0; qt < NQT; ++qt) {
    const int t = UQ * qb + 32 * qt + l32;
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
  constexpr int NW = kPfWaves, NQT = kPfQueryTiles;
  const int g = a.hq / a.hkv;
  const int units = ((a.max_seq_len + 32 * NQT - 1) / (32 * NQT)) * g;
  const dim3 grid((units + NW - 1) / NW, a.hkv, a.n_seqs);
  if (a.d == 128)
    hipLaunchKernelGGL((attn_prefill_kernel<128, NW, NQT>), grid, dim3(64 * NW), 0, st, a);
  else
    hipLaunchKernelGGL((attn_prefill_kernel<64, NW, NQT>), grid, dim3(64 * NW), 0, st, a);
  return hipGetLastError();
}

}  // namespace sevo
