// Paged GQA split-KV decode attention for gfx950 (one query token per
// candidate), plus the cross-split combine.
//
// Work decomposition: one 256-thread workgroup per (kv head, split, candidate).
// A split is a run of `chunk` logical pages of the candidate; its four waves
// take every fourth page, each keeping its own online-softmax state for the
// G = hq / hkv query heads that share the kv head, and merge through LDS at the
// end.  The combine kernel merges the splits of a (candidate, head) in split
// order, so results are deterministic and independent of the physical page
// order.  Groups of 4 or more heads run on the matrix cores (the second split
// kernel below); groups of 1 or 2 heads use vector dot products:
//
// Per page and wave (tile = 16 tokens x D dims, 4 KB at D = 128; the K and V
// tiles of a (page, kv head) are adjacent in the pool, so each page is one
// contiguous 8 KB read, measured about 2% faster than separate K and V pools):
//   QK  the K tile is stored in blocks of 32 dims ([D/32][16 tokens][32]), so
//       load ii reads block ii as one contiguous 1 KB wavefront access; lane
//       (t = lane/4, u = lane%4) gets dims 32 ii + 8u .. +7 of key t and forms
//       G partial dot products with v_dot2
//       (bf16 pairs, fp32 accumulate), and a 2-step DPP quad reduction
//       completes the score.  Scores are pre-scaled by scale*log2(e) so exp2
//       is used.
//   softmax  page max over the 16 tokens with register-only cross-lane ops
//       (DPP row rotates, permlane16/32 swaps); running max, rescale factor
//       and p = exp2(s - m) per head (wave-uniform max).
//   P   p is split into bf16 hi + lo parts (p = hi + lo to ~2^-17 relative,
//       so the softmax weights keep fp32-level accuracy through the bf16 dot
//       products); lanes holding token t (u == 0) write both to a per-wave LDS
//       strip and every lane reads the 8 values of its token half as packed
//       words.
//   PV  the V tile is dim-major [D][16] so one 32-bit word holds two tokens of
//       one dim: lane (dim 32*ii + lane/2, token half lane%2) accumulates
//       hi . v + lo . v with v_dot2 over token pairs.  Each 16-byte V load is
//       one contiguous 1 KB wavefront access.
// Loads for the wave's next two pages are issued before the current page is
// consumed (three register page buffers; two for G = 8, where registers are
// short).  A split spans at most 512 pages, so each wave's page ids fit one
// per lane in two registers, read out with readlane inside the loop.
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace sevo {

template <int D>
struct PageRegs {
  u32x4 k[D / 32];
  u32x4 v[D / 32];
};

// One K tile and one V tile of a page, read with raw buffer loads: the tile
// base goes into a wave-uniform buffer descriptor (scalar registers) and each
// lane's byte offset inside the tile is a fixed register, so the page loop
// does no vector address arithmetic.  A descriptor with zero records (a page
// id outside the pool) makes every load return zero without touching memory.
// Cache policy: streaming (nt), the KV cache is read once per step.
template <int D>
__device__ __forceinline__ void load_page(PageRegs<D>& r, const char* kt, const char* vt,
                                          int nrec, uint32_t koff, uint32_t voff) {
  constexpr int NI = D / 32;
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(kt), 0, nrec, 0x00020000);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(vt), 0, nrec, 0x00020000);
#pragma unroll
  for (int ii = 0; ii < NI; ++ii)
    r.k[ii] = __builtin_amdgcn_raw_buffer_load_b128(rk, (int)koff, ii * 1024, 2);
#pragma unroll
  for (int ii = 0; ii < NI; ++ii)
    r.v[ii] = __builtin_amdgcn_raw_buffer_load_b128(rv, (int)voff, ii * 1024, 2);
}

template <int D, int G>
__global__ __launch_bounds__(256, (G <= 4 ? 2 : 1)) void attn_split_kernel(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ kvpool,
    const int32_t* __restrict__ page_table, int max_pages,
    int num_pages32, const int32_t* __restrict__ seq_lens, int len_add, int hkv, int chunk, int S,
    float qk_scale_log2, float* __restrict__ part_ml, float* __restrict__ part_acc) {
  constexpr int NI = D / 32;
  // Grid (kv head, split, candidate): workgroups are dealt round-robin to the
  // 8 XCDs by linear id, so with 8 kv heads each XCD streams one head of every
  // candidate (equal work per XCD), and the splits of a candidate run side by
  // side (measured best among the orders of the three indices).
  const int c = blockIdx.x;
  const int s = blockIdx.y;
  const int i = blockIdx.z;
  const int hq = hkv * G;
  int len = seq_lens[i] + len_add;
  len = len < 0 ? 0 : (len > max_pages * kPage ? max_pages * kPage : len);
  const int npg = (len + kPage - 1) / kPage;
  const int pbeg = s * chunk;
  if (pbeg >= npg) return;  // empty split: the combine pass skips it
  const int pend = min(npg, pbeg + chunk);

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int t = lane >> 2, u = lane & 3;   // QK layout
  const int dl = lane >> 1, h = lane & 1;  // PV layout

  __shared__ __align__(16) bf16_t p_lds[4][2][G][kPage];  // [wave][hi|lo][head][token]
  __shared__ float w_m[4][G], w_l[4][G];
  __shared__ float w_acc[4][G][D];

  // q fragments of the G heads for this lane's dims
  uint32_t qf[G][NI][4];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    const bf16_t* qh = q + ((size_t)i * hq + (size_t)c * G + j) * D;
#pragma unroll
    for (int ii = 0; ii < NI; ++ii) {
      u32x4 w = *reinterpret_cast<const u32x4*>(qh + (u + 4 * ii) * 8);
      qf[j][ii][0] = w.x; qf[j][ii][1] = w.y; qf[j][ii][2] = w.z; qf[j][ii][3] = w.w;
    }
  }

  float m_run[G], l_run[G], acc[G][NI];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    m_run[j] = -INFINITY;
    l_run[j] = 0.f;
#pragma unroll
    for (int ii = 0; ii < NI; ++ii) acc[j][ii] = 0.f;
  }

  // The wave's page ids (at most 128: a split spans at most 512 pages) sit one
  // per lane in two registers; readlane turns each into a scalar with no
  // memory latency in the page loop.  Ids outside [0, num_pages) become -1
  // (the page is skipped).
  const int32_t* ptr = page_table + (size_t)i * max_pages;
  const int my_pages = (pend - (pbeg + wave) + 3) >> 2;
  int idv0 = -1, idv1 = -1;
  if (lane < my_pages) {
    const int id = ptr[pbeg + wave + 4 * lane];
    idv0 = (id >= 0 && id < num_pages32) ? id : -1;
  }
  if (lane + 64 < my_pages) {
    const int id = ptr[pbeg + wave + 4 * (lane + 64)];
    idv1 = (id >= 0 && id < num_pages32) ? id : -1;
  }
  auto page_id = [&](int k) -> int {
    const int kk = k < my_pages ? k : my_pages - 1;
    return kk < 64 ? __builtin_amdgcn_readlane(idv0, kk) : __builtin_amdgcn_readlane(idv1, kk - 64);
  };
  constexpr uint32_t kTileBytes = kPage * D * 2;
  const char* kv8 = reinterpret_cast<const char*>(kvpool);
  // lane byte offsets inside a tile: K block ii, token t, dims 8u..8u+7 of the
  // block; V dims 32 ii + dl, token half h
  const uint32_t koff = (uint32_t)(t * 64 + u * 16);
  const uint32_t voff = (uint32_t)(dl * kPage * 2 + h * 16);
#define SEVO_LOAD(BUF, K)                                                              \
  {                                                                                    \
    const int id_ = page_id(K);                                                        \
    const size_t tb_ = id_ < 0 ? 0 : ((size_t)id_ * hkv + c) * 2 * kTileBytes;        \
    load_page<D>(BUF, kv8 + tb_, kv8 + tb_ + kTileBytes, id_ < 0 ? 0 : (int)kTileBytes, \
                 koff, voff);                                                          \
  }

  // One page of the wave.  FULL: all 16 slots hold keys (no masking); else
  // `valid` keys (0 for a page id outside the pool).  The running max of each
  // head is wave-uniform, so the rescale of the accumulators is a uniform
  // branch taken only when a page raises the max.
  auto consume = [&](const PageRegs<D>& r, auto full_tag, int valid) {
    constexpr bool FULL = decltype(full_tag)::value;
    float sc[G];
#pragma unroll
    for (int j = 0; j < G; ++j) {
      float a = 0.f;
#pragma unroll
      for (int ii = 0; ii < NI; ++ii) {
        a = dot2_bf16(r.k[ii].x, qf[j][ii][0], a);
        a = dot2_bf16(r.k[ii].y, qf[j][ii][1], a);
        a = dot2_bf16(r.k[ii].z, qf[j][ii][2], a);
        a = dot2_bf16(r.k[ii].w, qf[j][ii][3], a);
      }
      a = quad_sum(a) * qk_scale_log2;
      if constexpr (FULL) sc[j] = a;
      else sc[j] = (t < valid) ? a : -INFINITY;
    }
#pragma unroll
    for (int j = 0; j < G; ++j) {
      const float pm = quads_max(sc[j]);  // the 4 lanes of a quad hold equal scores
      if (pm > m_run[j]) {
        const float alpha = __builtin_amdgcn_exp2f(m_run[j] - pm);  // 0 on the first page
        l_run[j] *= alpha;
#pragma unroll
        for (int ii = 0; ii < NI; ++ii) acc[j][ii] *= alpha;
        m_run[j] = pm;
      }
      const float p = m_run[j] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sc[j] - m_run[j]);
      l_run[j] += p;
      const __bf16 ph = (__bf16)p;
      const __bf16 pl = (__bf16)(p - (float)ph);
      if (u == 0) {
        p_lds[wave][0][j][t] = __builtin_bit_cast(bf16_t, ph);
        p_lds[wave][1][j][t] = __builtin_bit_cast(bf16_t, pl);
      }
    }
    // lanes read p values written by other lanes of the wave: order the LDS
    // stores before the loads for the compiler (the hardware keeps one wave's
    // LDS operations in order)
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    u32x4 pw[G], pwl[G];
#pragma unroll
    for (int j = 0; j < G; ++j) {
      pw[j] = *reinterpret_cast<const u32x4*>(&p_lds[wave][0][j][h * 8]);
      pwl[j] = *reinterpret_cast<const u32x4*>(&p_lds[wave][1][j][h * 8]);
    }
    u32x4 vv[NI];
#pragma unroll
    for (int ii = 0; ii < NI; ++ii) vv[ii] = r.v[ii];
    if constexpr (!FULL) {
      // slots past the last key may hold anything (even NaN patterns): zero them
      const int t0 = h * 8;
#pragma unroll
      for (int ii = 0; ii < NI; ++ii) {
        vv[ii].x = (t0 + 0 >= valid) ? 0u : ((t0 + 1 >= valid) ? (vv[ii].x & 0xFFFFu) : vv[ii].x);
        vv[ii].y = (t0 + 2 >= valid) ? 0u : ((t0 + 3 >= valid) ? (vv[ii].y & 0xFFFFu) : vv[ii].y);
        vv[ii].z = (t0 + 4 >= valid) ? 0u : ((t0 + 5 >= valid) ? (vv[ii].z & 0xFFFFu) : vv[ii].z);
        vv[ii].w = (t0 + 6 >= valid) ? 0u : ((t0 + 7 >= valid) ? (vv[ii].w & 0xFFFFu) : vv[ii].w);
      }
    }
#pragma unroll
    for (int j = 0; j < G; ++j) {
#pragma unroll
      for (int ii = 0; ii < NI; ++ii) {
        float a = acc[j][ii];
        a = dot2_bf16(vv[ii].x, pwl[j].x, a);
        a = dot2_bf16(vv[ii].y, pwl[j].y, a);
        a = dot2_bf16(vv[ii].z, pwl[j].z, a);
        a = dot2_bf16(vv[ii].w, pwl[j].w, a);
        a = dot2_bf16(vv[ii].x, pw[j].x, a);
        a = dot2_bf16(vv[ii].y, pw[j].y, a);
        a = dot2_bf16(vv[ii].z, pw[j].z, a);
        a = dot2_bf16(vv[ii].w, pw[j].w, a);
        acc[j][ii] = a;
      }
    }
  };
  // dispatch a page: full pages take the unmasked path
  auto consume_page = [&](const PageRegs<D>& r, int k) {
    const int pg = pbeg + wave + 4 * k;
    int valid = len - pg * kPage;
    valid = valid > kPage ? kPage : valid;
    if (page_id(k) < 0) valid = 0;
    if (valid == kPage) consume(r, std::true_type{}, kPage);
    else consume(r, std::false_type{}, valid);
  };

  if (my_pages > 0) {
    int k = 0;  // this wave's page index: logical page pbeg + wave + 4k
    if constexpr (G <= 4) {
      // three page buffers: while page k is consumed, pages k+1 and k+2 are in
      // flight (16 KB per wave at D = 128)
      PageRegs<D> A, B, C;
      SEVO_LOAD(A, 0)
      SEVO_LOAD(B, 1)
      while (true) {
        SEVO_LOAD(C, k + 2)
        consume_page(A, k);
        if (++k >= my_pages) break;
        SEVO_LOAD(A, k + 2)
        consume_page(B, k);
        if (++k >= my_pages) break;
        SEVO_LOAD(B, k + 2)
        consume_page(C, k);
        if (++k >= my_pages) break;
      }
    } else {
      // two page buffers (registers are short at G = 8)
      PageRegs<D> A, B;
      SEVO_LOAD(A, 0)
      while (true) {
        SEVO_LOAD(B, k + 1)
        consume_page(A, k);
        if (++k >= my_pages) break;
        SEVO_LOAD(A, k + 1)
        consume_page(B, k);
        if (++k >= my_pages) break;
      }
    }
  }

#undef SEVO_LOAD
  // finish this wave: sum V partials over the two token halves, l over tokens
#pragma unroll
  for (int j = 0; j < G; ++j) {
#pragma unroll
    for (int ii = 0; ii < NI; ++ii) acc[j][ii] += dpp<kDppQuadXor1>(acc[j][ii]);
    l_run[j] = quads_sum(l_run[j]);  // over the 16 tokens (lanes of one quad agree)
  }
  if (lane == 0) {
#pragma unroll
    for (int j = 0; j < G; ++j) {
      w_m[wave][j] = m_run[j];
      w_l[wave][j] = l_run[j];
    }
  }
  if (h == 0) {
#pragma unroll
    for (int j = 0; j < G; ++j)
#pragma unroll
      for (int ii = 0; ii < NI; ++ii) w_acc[wave][j][32 * ii + dl] = acc[j][ii];
  }
  __syncthreads();

  // merge the four waves (fixed order) and store this split's partial
  for (int idx = threadIdx.x; idx < G * D; idx += 256) {
    const int j = idx / D;
    const int e = idx - j * D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, w_m[w][j]);
    float L = 0.f, A = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float mw = w_m[w][j];
      if (mw != -INFINITY) {
        const float f = exp2f(mw - M);
        L += w_l[w][j] * f;
        A += w_acc[w][j][e] * f;
      }
    }
    const size_t slot = ((size_t)i * hq + (size_t)c * G + j) * S + s;
    part_acc[slot * D + e] = A;
    if (e == 0) {
      part_ml[slot * 2] = M;
      part_ml[slot * 2 + 1] = L;
    }
  }
}

// The same split attention for groups of G >= 4 query heads per kv head, on
// the matrix cores.  With G heads a page is a small dense product (16 tokens
// x G heads x D dims): at G = 8 the vector dot products above cannot keep up
// with HBM (measured 2.75 TB/s against 6.15 here), and at G = 4 this variant
// is still a few percent faster; per page and wave:
//   QK  S = K Q^T with v_mfma_f32_16x16x32_bf16 over the D/32 dim blocks
//       (A = the K tile, rows = tokens; B = the q fragments, columns = heads,
//       columns >= G are zero): lane (head l % 16, token group l / 16) gets
//       the scores of tokens 4 (l / 16) + 0..3 of its head.
//   softmax  page max per head over the 4 token groups (two permlane swaps),
//       lazy running max: the accumulators are rescaled only when a page
//       raises a head's max by more than 2^kLazyRescaleLog2, which after the
//       first pages is rare; p = exp2(s - m) <= 2^kLazyRescaleLog2.
//   P   p = hi + lo (bf16 each, ~2^-17 relative), written to a per-wave LDS
//       strip [hi|lo][head][token] and read back as the B operand of PV.
//   PV  O^T = V^T P^T with one 16x16x32 MFMA per 16-dim block whose 32-deep
//       k axis is [tokens of P hi | tokens of P lo] against the V tile twice,
//       so one instruction takes both halves; the output lane holds its own
//       head (l % 16) and dims 16 b + 4 (l / 16) + 0..3, so the rescale needs
//       no data from other lanes.
// Loads of the wave's next two pages are in flight while a page is consumed.
constexpr float kLazyRescaleLog2 = 8.f;

template <int D, int G>
__global__ __launch_bounds__(256, 2) void attn_split_mfma_kernel(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ kvpool,
    const int32_t* __restrict__ page_table, int max_pages,
    int num_pages32, const int32_t* __restrict__ seq_lens, int len_add, int hkv, int chunk, int S,
    float qk_scale_log2, float* __restrict__ part_ml, float* __restrict__ part_acc) {
  static_assert(G >= 4 && G <= 16, "one 16-column MFMA tile of heads");
  constexpr int NI = D / 32;  // 32-dim blocks of K
  constexpr int NB = D / 16;  // 16-dim blocks of the output
  const int c = blockIdx.x;
  const int s = blockIdx.y;
  const int i = blockIdx.z;
  const int hq = hkv * G;
  int len = seq_lens[i] + len_add;
  len = len < 0 ? 0 : (len > max_pages * kPage ? max_pages * kPage : len);
  const int npg = (len + kPage - 1) / kPage;
  const int pbeg = s * chunk;
  if (pbeg >= npg) return;  // empty split: the combine pass skips it
  const int pend = min(npg, pbeg + chunk);

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15;  // head (QK / PV columns), token (K rows), dim (V rows)
  const int grp = lane >> 4;

  __shared__ __align__(16) bf16_t p_lds[4][2][16][kPage];  // [wave][hi|lo][head][token]
  __shared__ float w_m[4][G], w_l[4][G];
  __shared__ float w_acc[4][G][D];

  // B operand of QK: head `col`, dims 32 ii + 8 grp .. +7 (zero for col >= G)
  bf16x8v qf[NI];
#pragma unroll
  for (int ii = 0; ii < NI; ++ii) {
    u32x4 w = u32x4{0u, 0u, 0u, 0u};
    if (col < G)
      w = *reinterpret_cast<const u32x4*>(q + ((size_t)i * hq + (size_t)c * G + col) * D +
                                          32 * ii + 8 * grp);
    qf[ii] = __builtin_bit_cast(bf16x8v, w);
  }
  float m_run = -INFINITY, l_run = 0.f;
  f32x4 acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) acc[b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int32_t* ptr = page_table + (size_t)i * max_pages;
  const int my_pages = (pend - (pbeg + wave) + 3) >> 2;
  int idv0 = -1, idv1 = -1;
  if (lane < my_pages) {
    const int id = ptr[pbeg + wave + 4 * lane];
    idv0 = (id >= 0 && id < num_pages32) ? id : -1;
  }
  if (lane + 64 < my_pages) {
    const int id = ptr[pbeg + wave + 4 * (lane + 64)];
    idv1 = (id >= 0 && id < num_pages32) ? id : -1;
  }
  auto page_id = [&](int k) -> int {
    const int kk = k < my_pages ? k : my_pages - 1;
    return kk < 64 ? __builtin_amdgcn_readlane(idv0, kk) : __builtin_amdgcn_readlane(idv1, kk - 64);
  };
  constexpr uint32_t kTileBytes = kPage * D * 2;
  const char* kv8 = reinterpret_cast<const char*>(kvpool);
  // K: block ii, token col, dims 8 grp..+7; V: dim 16 b + col, tokens 8 (grp & 1)..+7
  const uint32_t koff = (uint32_t)(col * 64 + grp * 16);
  const uint32_t voff = (uint32_t)(col * kPage * 2 + (grp & 1) * 16);
  struct Regs {
    u32x4 k[NI];
    u32x4 v[NB];
  };
  auto load = [&](Regs& r, int k) {
    const int id = page_id(k);
    const size_t tb = id < 0 ? 0 : ((size_t)id * hkv + c) * 2 * kTileBytes;
    const int nrec = id < 0 ? 0 : (int)kTileBytes;
    const __amdgpu_buffer_rsrc_t rk =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(kv8 + tb), 0, nrec, 0x00020000);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(kv8 + tb + kTileBytes), 0, nrec, 0x00020000);
#pragma unroll
    for (int ii = 0; ii < NI; ++ii)
      r.k[ii] = __builtin_amdgcn_raw_buffer_load_b128(rk, (int)koff, ii * 1024, 2);
#pragma unroll
    for (int b = 0; b < NB; ++b)
      r.v[b] = __builtin_amdgcn_raw_buffer_load_b128(rv, (int)voff, b * 16 * kPage * 2, 2);
  };

  auto consume = [&](const Regs& r, int k) {
    const int pg = pbeg + wave + 4 * k;
    int valid = len - pg * kPage;
    valid = valid > kPage ? kPage : valid;
    if (page_id(k) < 0) valid = 0;
    f32x4 sc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ii = 0; ii < NI; ++ii)
      sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8v, r.k[ii]), qf[ii],
                                                   sc, 0, 0, 0);
    float z[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      z[e] = (4 * grp + e < valid) ? sc[e] * qk_scale_log2 : -INFINITY;
    float pm = fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3]));
    pm = xor32_max(xor16_max(pm));
    // lazy running max (a wave-uniform branch, rarely taken after the first pages)
    const bool raise = pm > m_run + kLazyRescaleLog2;
    if (__builtin_amdgcn_ballot_w64(raise)) {
      const float mn = raise ? pm : m_run;
      const float alpha = raise ? __builtin_amdgcn_exp2f(m_run - mn) : 1.f;  // 0 on the first page
      l_run *= alpha;
#pragma unroll
      for (int b = 0; b < NB; ++b) acc[b] *= alpha;
      m_run = mn;
    }
    uint32_t hi[2], lo[2];
#pragma unroll
    for (int e = 0; e < 4; e += 2) {
      const float p0 = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(z[e] - m_run);
      const float p1 = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(z[e + 1] - m_run);
      l_run += p0 + p1;
      const __bf16 h0 = (__bf16)p0, h1 = (__bf16)p1;
      const __bf16 q0 = (__bf16)(p0 - (float)h0), q1 = (__bf16)(p1 - (float)h1);
      hi[e / 2] = (uint32_t)__builtin_bit_cast(uint16_t, h0) |
                  ((uint32_t)__builtin_bit_cast(uint16_t, h1) << 16);
      lo[e / 2] = (uint32_t)__builtin_bit_cast(uint16_t, q0) |
                  ((uint32_t)__builtin_bit_cast(uint16_t, q1) << 16);
    }
    *reinterpret_cast<uint2*>(&p_lds[wave][0][col][4 * grp]) = uint2{hi[0], hi[1]};
    *reinterpret_cast<uint2*>(&p_lds[wave][1][col][4 * grp]) = uint2{lo[0], lo[1]};
    // lanes read p values written by other lanes of the wave: order the LDS
    // stores before the loads for the compiler (the hardware keeps one wave's
    // LDS operations in order)
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const bf16x8v pb = __builtin_bit_cast(
        bf16x8v, *reinterpret_cast<const u32x4*>(&p_lds[wave][grp >> 1][col][8 * (grp & 1)]));
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      u32x4 vv = r.v[b];
      if (valid < kPage) {
        // slots past the last key may hold anything (even NaN patterns): zero them
        const int t0 = 8 * (grp & 1);
        vv.x = (t0 + 0 >= valid) ? 0u : ((t0 + 1 >= valid) ? (vv.x & 0xFFFFu) : vv.x);
        vv.y = (t0 + 2 >= valid) ? 0u : ((t0 + 3 >= valid) ? (vv.y & 0xFFFFu) : vv.y);
        vv.z = (t0 + 4 >= valid) ? 0u : ((t0 + 5 >= valid) ? (vv.z & 0xFFFFu) : vv.z);
        vv.w = (t0 + 6 >= valid) ? 0u : ((t0 + 7 >= valid) ? (vv.w & 0xFFFFu) : vv.w);
      }
      acc[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8v, vv), pb, acc[b],
                                                       0, 0, 0);
    }
  };

  if (my_pages > 0) {
    int k = 0;  // this wave's page index: logical page pbeg + wave + 4k
    Regs A, B, C;
    load(A, 0);
    load(B, 1);
    while (true) {
      load(C, k + 2);
      consume(A, k);
      if (++k >= my_pages) break;
      load(A, k + 2);
      consume(B, k);
      if (++k >= my_pages) break;
      load(B, k + 2);
      consume(C, k);
      if (++k >= my_pages) break;
    }
  }

  // finish this wave: l over the 4 token groups; the accumulators already
  // hold full sums over the tokens
  l_run = xor32_sum(xor16_sum(l_run));
  if (grp == 0 && col < G) {
    w_m[wave][col] = m_run;
    w_l[wave][col] = l_run;
  }
  if (col < G) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int e = 0; e < 4; ++e) w_acc[wave][col][16 * b + 4 * grp + e] = acc[b][e];
  }
  __syncthreads();

  // merge the four waves (fixed order) and store this split's partial
  for (int idx = threadIdx.x; idx < G * D; idx += 256) {
    const int j = idx / D;
    const int e = idx - j * D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, w_m[w][j]);
    float L = 0.f, Acc = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float mw = w_m[w][j];
      if (mw != -INFINITY) {
        const float f = exp2f(mw - M);
        L += w_l[w][j] * f;
        Acc += w_acc[w][j][e] * f;
      }
    }
    const size_t slot = ((size_t)i * hq + (size_t)c * G + j) * S + s;
    part_acc[slot * D + e] = Acc;
    if (e == 0) {
      part_ml[slot * 2] = M;
      part_ml[slot * 2 + 1] = L;
    }
  }
}

// Merge the non-empty splits of one (candidate, query head), in split order.
template <int D>
__global__ __launch_bounds__(64) void attn_combine_kernel(const float* __restrict__ part_ml,
                                                          const float* __restrict__ part_acc,
                                                          const int32_t* __restrict__ seq_lens,
                                                          int len_add, int max_pages, int chunk, int S, int hq,
                                                          bf16_t* __restrict__ out, int out_tiled) {
  constexpr int E = D / 64;
  const int j = blockIdx.x;
  const int i = blockIdx.y;
  int len = seq_lens[i] + len_add;
  len = len < 0 ? 0 : (len > max_pages * kPage ? max_pages * kPage : len);
  const int npg = (len + kPage - 1) / kPage;
  int ns = (npg + chunk - 1) / chunk;
  ns = ns > S ? S : ns;
  const size_t base = ((size_t)i * hq + j) * S;
  // splits in order, four splits' loads issued together (a load per split
  // and pass would wait out one memory latency each)
  float M = -INFINITY;
  for (int s0 = 0; s0 < ns; s0 += 4) {
    float mm[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) mm[j] = s0 + j < ns ? part_ml[(base + s0 + j) * 2] : -INFINITY;
#pragma unroll
    for (int j = 0; j < 4; ++j) M = fmaxf(M, mm[j]);
  }
  float L = 0.f, a[E];
#pragma unroll
  for (int e = 0; e < E; ++e) a[e] = 0.f;
  for (int s0 = 0; s0 < ns; s0 += 4) {
    float ms[4], ls[4], ac[4][E];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      ms[j] = -INFINITY;
      if (s0 + j < ns) {
        ms[j] = part_ml[(base + s0 + j) * 2];
        ls[j] = part_ml[(base + s0 + j) * 2 + 1];
#pragma unroll
        for (int e = 0; e < E; ++e) ac[j][e] = part_acc[(base + s0 + j) * D + threadIdx.x + 64 * e];
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (ms[j] == -INFINITY) continue;
      const float f = exp2f(ms[j] - M);
      L += ls[j] * f;
#pragma unroll
      for (int e = 0; e < E; ++e) a[e] += ac[j][e] * f;
    }
  }
  const float inv = L > 0.f ? 1.0f / L : 0.f;
  // row-major [n][hq][D], or the tiled activation layout of [n][hq D] (the
  // output projection's input)
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int c = j * D + threadIdx.x + 64 * e;
    const size_t off = out_tiled ? act_tile_offset(i, c, hq * D) : (size_t)i * hq * D + c;
    out[off] = f32_to_bf16(a[e] * inv);
  }
}

template <int D, int G>
static hipError_t launch_attn_t(const AttnArgs& a, hipStream_t st) {
  const float log2e = 1.4426950408889634f;
  if (a.ev_begin) (void)hipEventRecord(a.ev_begin, st);
  // G >= 4 heads per kv head: the matrix-core variant
  using SplitFn = void (*)(const bf16_t*, const bf16_t*, const int32_t*, int, int, const int32_t*,
                           int, int, int, int, float, float*, float*);
  SplitFn fn;
  if constexpr (G >= 4) fn = attn_split_mfma_kernel<D, G>;
  else fn = attn_split_kernel<D, G>;
  hipLaunchKernelGGL(fn, dim3(a.hkv, a.num_splits, a.n), dim3(256), 0, st,
                     a.q, a.kv_pool, a.page_table, a.max_pages,
                     (int)(a.num_pages < 0x7FFFFFFF ? a.num_pages : 0x7FFFFFFF), a.seq_lens,
                     a.len_add, a.hkv, a.chunk, a.num_splits, a.scale * log2e, a.part_ml, a.part_acc);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.ev_mid) (void)hipEventRecord(a.ev_mid, st);
  hipLaunchKernelGGL((attn_combine_kernel<D>), dim3(a.hq, a.n), dim3(64), 0, st, a.part_ml,
                     a.part_acc, a.seq_lens, a.len_add, a.max_pages, a.chunk, a.num_splits, a.hq, a.out,
                     a.out_tiled);
  e = hipGetLastError();
  if (e == hipSuccess && a.ev_end) (void)hipEventRecord(a.ev_end, st);
  return e;
}

hipError_t launch_attn_decode(const AttnArgs& a, hipStream_t st) {
  if (a.n == 0) return hipSuccess;
  const int g = a.hq / a.hkv;
#define SEVO_ATTN_CASE(DD, GG) \
  if (a.d == DD && g == GG) return launch_attn_t<DD, GG>(a, st);
  SEVO_ATTN_CASE(128, 1)
  SEVO_ATTN_CASE(128, 2)
  SEVO_ATTN_CASE(128, 4)
  SEVO_ATTN_CASE(128, 8)
  SEVO_ATTN_CASE(64, 1)
  SEVO_ATTN_CASE(64, 2)
  SEVO_ATTN_CASE(64, 4)
  SEVO_ATTN_CASE(64, 8)
#undef SEVO_ATTN_CASE
  return hipErrorInvalidValue;
}

}  // namespace sevo
