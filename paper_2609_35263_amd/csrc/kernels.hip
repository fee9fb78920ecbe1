// gfx950 (CDNA4) kernels of libwavepp_attn: K/V append into reserved pages, chunked-prefill
// attention over paged K/V with bf16 MFMA, and the merge of key-range splits.
//
// Attention layout (one workgroup = 8 waves = one work item of up to 256 query rows; one workgroup
// per CU, two waves per SIMD.  A 4-wave form with 128-row items and 64-key tiles runs two
// workgroups per CU for waves whose (request, KV head) pairs have at most 128 rows):
//   * Rows are (token, head-in-group) pairs of one (request, KV head): row = token * G + h, so the
//     G query heads that share a KV head share every K/V tile loaded into LDS.
//   * Each wave owns 32 rows.  Logits are computed transposed, S^T = K Q^T, with
//     v_mfma_f32_32x32x16_bf16: the K tile (from LDS) is the A operand and the wave's Q rows
//     (kept in registers for the whole loop) are the B operand.  In the 32x32 accumulator each
//     lane then holds 16 logits of ONE query row, so the softmax row max / row sum are in-lane
//     reductions plus a single exchange between the two half-waves.
//   * The exponentiated probabilities are rounded to bf16 and fed straight back as the B operand
//     of O^T += V^T P^T: the key order inside that contraction is the order in which the
//     accumulator holds them.  V is staged in LDS row-major like K and read with gfx950's
//     transposing LDS load (ds_read_b64_tr_b16) in that matching order.
//   * K/V tiles of 128 keys (64 in the 4-wave form) are gathered from the pages named by the block
//     table with 16-byte loads (one page's head slice is contiguous), double-buffered in LDS: the
//     next tile's global loads are issued before the current tile's MFMAs and written to the other
//     buffer after.
//   * Online softmax in fp32 (exp2 with the log2(e) factor folded into the scale); masking is by
//     selection, and K/V rows past the request's last valid position are never loaded (their
//     addresses are clamped to the last valid row), so stale or NaN pool slots cannot leak into
//     the output.
#include <hip/hip_runtime.h>

#include "internal.h"

#include <algorithm>
#include <mutex>
#include <type_traits>

namespace wavepp {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ bool meta_ok(const DevPlan& p) {
  return p.hdr->magic == kMagic && p.hdr->serial == p.serial;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// ---------------------------------------------------------------------------------------------
// Append: token t of request r -> page bt[r][(p_r + i) / B], slot (p_r + i) % B, all KV heads.
// One workgroup moves kAppendTokens consecutive packed tokens; for each token its threads move the
// Hkv * (DK + DV) / 8 16-byte chunks (the workgroup has that many threads rounded up to a whole
// wave, at most 256).  The token's request and page are uniform across the
// workgroup, so they are looked up once, with scalar loads through the constant address space
// (the kernel never writes the metadata).
// ---------------------------------------------------------------------------------------------
constexpr int kAppendTokens = 8;

template <typename T>
__device__ __forceinline__ T const_load(const T* ptr) {
  return *((const __attribute__((address_space(4))) T*)(ptr));
}

template <int DK, int DV>
__global__ __launch_bounds__(256) void append_kernel(DevPlan p, const uint4* __restrict__ k_new,
                                                     const uint4* __restrict__ v_new, uint4* __restrict__ k_pool,
                                                     uint4* __restrict__ v_pool) {
  if (!meta_ok(p)) return;
  constexpr int KC = DK / 8, VC = DV / 8, UC = KC + VC;
  const int Hkv = p.num_kv_heads;
  const int per_tok = Hkv * UC;
  const int B = p.page_size;
  const int64_t T = p.total_tokens;
  const int64_t t0 = int64_t(blockIdx.x) * kAppendTokens;
  // request holding token t0: the last r with cu_r <= t0 (requests with no chunk share cu with the next)
  int lo = 0, hi = p.num_requests - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (const_load(&p.reqs[mid].cu) <= t0) lo = mid; else hi = mid - 1;
  }
  int r = lo;
#pragma unroll
  for (int i = 0; i < kAppendTokens; ++i) {
    const int64_t t = t0 + i;
    if (t >= T) break;
    while (r + 1 < p.num_requests && const_load(&p.reqs[r + 1].cu) <= t) ++r;
    const ReqMeta* rq = &p.reqs[r];
    const int pos = const_load(&rq->prefix) + int(t - const_load(&rq->cu));
    const int64_t page = const_load(&p.bt[const_load(&rq->bt_row) + pos / B]);
    const int slot = pos % B;
    for (int u = threadIdx.x; u < per_tok; u += blockDim.x) {
      const int h = u / UC;
      const int c = u - h * UC;
      if (c < KC) {
        k_pool[((page * Hkv + h) * B + slot) * KC + c] = k_new[(t * Hkv + h) * KC + c];
      } else {
        const int cv = c - KC;
        v_pool[((page * Hkv + h) * B + slot) * VC + cv] = v_new[(t * Hkv + h) * VC + cv];
      }
    }
  }
}

// ---------------------------------------------------------------------------------------------
// Grouped-query attention, head dim D (64 or 128), page size PAGE (16 or 64).
// ---------------------------------------------------------------------------------------------
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// Both halves of the wave receive max / sum of their value and the other half's value for the
// same query row (lanes l and l ^ 32).
__device__ __forceinline__ float halves_max(float x) {
  const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(s[0]), __uint_as_float(s[1]));
}
__device__ __forceinline__ float halves_sum(float x) {
  const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(s[0]) + __uint_as_float(s[1]);
}

// Transposing LDS read: within each group of 16 lanes, lane i receives element i%4 of the 8 bytes
// addressed by lanes 4m + i/4, m = 0..3.
__device__ __forceinline__ bf16x4 lds_read_tr(const __bf16* p) {
  const i16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
  return __builtin_bit_cast(bf16x4, r);
}

template <int D, int PAGE, int NW>
__global__ __launch_bounds__(NW * 64, NW == 4 ? 2 : 1) void attn_gqa_kernel(DevPlan p, const __bf16* __restrict__ q,
                                                          const __bf16* __restrict__ kpool,
                                                          const __bf16* __restrict__ vpool, __bf16* __restrict__ out,
                                                          float* __restrict__ lse_out) {
  constexpr int KT = NW == 4 ? kKvTile / 2 : kKvTile;   // keys per tile (4-wave form: two workgroups per CU)
  constexpr int NKB = KT / 32;         // 32-key blocks per tile
  constexpr int NT = NW * 64;          // threads per workgroup; NW waves x 32 query rows
  constexpr int KSTR = D + 8;          // K rows in LDS: 16-byte reads of 8 rows land on distinct banks
  constexpr int VSTR = D + 32;         // V rows in LDS: transposed reads of 4 rows x 2 groups x 32 bytes on distinct banks
  constexpr int CH = D / 8;            // 16-byte chunks per key row
  constexpr int LOADS = KT * CH / NT;  // chunks per thread per tile, for K and for V alike
  constexpr int PPT = (PAGE >= KT) ? 1 : KT / PAGE;   // pages touched by one tile
  static_assert(LOADS >= 1 && LOADS * NT == KT * CH, "tile covered exactly");
  __shared__ __attribute__((aligned(16))) __bf16 ks[2][KT * KSTR];
  __shared__ __attribute__((aligned(16))) __bf16 vs[2][KT * VSTR];

  if (!meta_ok(p)) return;
  const WorkItem it = p.items[blockIdx.x];
  if (it.rows <= 0) return;
  const ReqMeta rm = p.reqs[it.req];
  const int Hq = p.num_q_heads, Hkv = p.num_kv_heads;
  const int G = Hq / Hkv;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, col = lane & 31, hf = lane >> 5;
  const int n_valid = rm.prefix + rm.chunk;
  const int32_t* __restrict__ bt = p.bt + rm.bt_row;
  const int64_t page_stride = int64_t(Hkv) * PAGE * D;
  const __bf16* __restrict__ kpool_h = kpool + int64_t(it.kv_head) * PAGE * D;
  const __bf16* __restrict__ vpool_h = vpool + int64_t(it.kv_head) * PAGE * D;

  // ---- this lane's query row -----------------------------------------------------------------
  const int lrow = wave * 32 + col;
  const bool row_ok = lrow < it.rows;
  const int prow = it.row0 + (row_ok ? lrow : 0);
  const int tok = prow / G;
  const int head = it.kv_head * G + (prow - tok * G);
  const int limit = rm.prefix + tok;                             // last key this row may see
  bf16x8 qf[D / 16];
  {
    const __bf16* qrow = q + (int64_t(rm.cu + tok) * Hq + head) * D + 8 * hf;
#pragma unroll
    for (int s = 0; s < D / 16; ++s) qf[s] = row_ok ? *reinterpret_cast<const bf16x8*>(qrow + 16 * s) : bf16x8{};
  }
  const int wrow0 = wave * 32;
  const bool wave_active = wrow0 < it.rows;
  const int wrow_last = min(it.rows, wrow0 + 32) - 1;
  const int wave_min_lim = rm.prefix + (it.row0 + wrow0) / G;
  const int wave_max_lim = rm.prefix + (it.row0 + max(wrow_last, wrow0)) / G;

  f32x16 oacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db) oacc[db] = f32x16{};
  float m_run = -INFINITY, l_run = 0.0f;
  const float sl2 = p.softmax_scale * kLog2e;

  // ---- K/V tile staging -----------------------------------------------------------------------
  // Thread tid moves 16-byte chunks c = tid + NT i of both the K and the V tile: key c / CH, chunk
  // c % CH; consecutive threads read consecutive 16 bytes of a page's contiguous head slice.  The
  // physical pages of a tile are looked up one tile ahead (uniform across the workgroup, hence
  // scalar loads) and the loads of tile t+1 are issued before the MFMAs of tile t.  A whole tile
  // uses offsets fixed per thread; in the last tile of a request, key positions past its last valid
  // slot are clamped to that slot: those rows are finite copies that the mask gives zero weight, so
  // stale or NaN pool slots are never read.
  const int last_block = (n_valid - 1) / PAGE;
  int ckey[LOADS], csub[LOADS];
  uint32_t coff[LOADS], cfull[LOADS];
#pragma unroll
  for (int i = 0; i < LOADS; ++i) {
    const int c = tid + NT * i;
    ckey[i] = c / CH;
    csub[i] = ckey[i] / PAGE;
    coff[i] = uint32_t((c % CH) * 8);
    cfull[i] = uint32_t(ckey[i] % PAGE) * D + coff[i];
  }
  u32x4 kreg[LOADS], vreg[LOADS];
  int pg_nxt[PPT];

#define WAVEPP_TILE_PAGES(tile_, pg_)                                                                     \
  _Pragma("unroll") for (int i_ = 0; i_ < PPT; ++i_) pg_[i_] = bt[min((tile_) * (KT / PAGE) + i_, last_block)];

#define WAVEPP_LOAD_TILE(tile_, pg_)                                                                      \
  {                                                                                                       \
    const int kbase_ = (tile_) * KT;                                                                      \
    if (kbase_ + KT <= n_valid) {                                                                         \
      _Pragma("unroll") for (int i_ = 0; i_ < LOADS; ++i_) {                                              \
        int page_ = pg_[0];                                                                               \
        _Pragma("unroll") for (int q_ = 1; q_ < PPT; ++q_) page_ = (csub[i_] == q_) ? pg_[q_] : page_;    \
        kreg[i_] = *reinterpret_cast<const u32x4*>(kpool_h + int64_t(page_) * page_stride + cfull[i_]);   \
        vreg[i_] = *reinterpret_cast<const u32x4*>(vpool_h + int64_t(page_) * page_stride + cfull[i_]);   \
      }                                                                                                   \
    } else {                                                                                              \
      _Pragma("unroll") for (int i_ = 0; i_ < LOADS; ++i_) {                                              \
        const int j_ = min(kbase_ + ckey[i_], n_valid - 1);                                               \
        const int sub_ = (j_ - kbase_) / PAGE;                                                            \
        int page_ = pg_[0];                                                                               \
        _Pragma("unroll") for (int q_ = 1; q_ < PPT; ++q_) page_ = (sub_ == q_) ? pg_[q_] : page_;        \
        const uint32_t off_ = uint32_t(j_ % PAGE) * D + coff[i_];                                         \
        kreg[i_] = *reinterpret_cast<const u32x4*>(kpool_h + int64_t(page_) * page_stride + off_);       \
        vreg[i_] = *reinterpret_cast<const u32x4*>(vpool_h + int64_t(page_) * page_stride + off_);       \
      }                                                                                                   \
    }                                                                                                     \
  }

#define WAVEPP_STORE_TILE(buf_)                                                                           \
  _Pragma("unroll") for (int i_ = 0; i_ < LOADS; ++i_) {                                                  \
    *reinterpret_cast<u32x4*>(&ks[buf_][ckey[i_] * KSTR + coff[i_]]) = kreg[i_];                          \
    *reinterpret_cast<u32x4*>(&vs[buf_][ckey[i_] * VSTR + coff[i_]]) = vreg[i_];                          \
  }

  // per-lane LDS read bases.  K (A operand of S^T = K Q^T): row col, elements 8*hf.. of each
  // 16-wide step.  V (A operand of O^T = V^T P^T, read transposed): within its 16-lane group, lane
  // j = lane % 16 addresses key 4*hf + j/4 and d = 16*((lane/16) % 2) + 4*(j%4) of a 16-key step.
  const int k_lane = col * KSTR + 8 * hf;
  const int v_lane = (4 * hf + (lane & 15) / 4) * VSTR + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  const int t_begin = it.kv_begin / KT;
  const int t_end = (it.kv_end + KT - 1) / KT;
  {
    int pg_cur[PPT];
    WAVEPP_TILE_PAGES(t_begin, pg_cur)
    WAVEPP_TILE_PAGES(t_begin + 1, pg_nxt)
    WAVEPP_LOAD_TILE(t_begin, pg_cur)
    WAVEPP_STORE_TILE(0)
  }
  __syncthreads();

  for (int tile = t_begin; tile < t_end; ++tile) {
    const int buf = (tile - t_begin) & 1;
    const bool has_next = tile + 1 < t_end;
    if (has_next) {
      WAVEPP_LOAD_TILE(tile + 1, pg_nxt)
      WAVEPP_TILE_PAGES(tile + 2, pg_nxt)
    }
    const int kbase = tile * KT;
    if (wave_active && kbase <= wave_max_lim) {
      // S^T[key][row] for the KT keys of the tile, as NKB 32-key blocks
      f32x16 sacc[NKB];
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) sacc[kb] = f32x16{};
      const __bf16* kl = &ks[buf][k_lane];
#pragma unroll
      for (int s = 0; s < D / 16; ++s)
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
          const bf16x8 kf = *reinterpret_cast<const bf16x8*>(kl + 32 * kb * KSTR + 16 * s);
          sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], sacc[kb], 0, 0, 0);
        }
      // keep four K fragment reads in flight ahead of the MFMAs that consume them
      __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
      for (int i = 0; i < (D / 16) * NKB - 4; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
      // accumulator element r of block kb holds key 32*kb + 8*(r/4) + 4*hf + (r%4)
      const bool need_mask = (kbase + KT - 1 > wave_min_lim) || (kbase + KT > it.kv_end);
      if (need_mask) {
        // key > limit or key >= kv_end  <=>  (key - kbase - 4 hf) > bound, one compare per element
        const int bound = min(limit, it.kv_end - 1) - kbase - 4 * hf;
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (32 * kb + 8 * (r >> 2) + (r & 3) > bound) sacc[kb][r] = -INFINITY;
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kb][r]);
      mx = halves_max(mx) * sl2;
      // The reference max only moves when the tile's max exceeds it by more than 2^8, so most tiles
      // skip rescaling the accumulators; probabilities stay below 256, which bf16/fp32 represent as
      // well as values below 1.  The final normalization uses the same reference.
      const bool bump = mx > m_run + 8.0f;
      const float m_new = bump ? mx : m_run;
      const float m_use = (m_new == -INFINITY) ? 0.0f : m_new;
      float rs = 0.0f;
      bf16x8 pb[2 * NKB];
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float e = fast_exp2(fmaf(sacc[kb][r], sl2, -m_use));
          rs += e;
          pb[2 * kb + (r >> 3)][r & 7] = static_cast<__bf16>(e);
        }
      rs = halves_sum(rs);
      if (__any(bump)) {
        const float alpha = fast_exp2(m_run - m_use);
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
      }
      l_run += rs;
      m_run = m_new;
      // O^T[d][row] += V^T[d][key] P^T[key][row]; step t covers keys 16t + 8*(e/4) + 4*hf + (e%4),
      // the order in which the S^T accumulator holds them
      const __bf16* vl = &vs[buf][v_lane];
#pragma unroll
      for (int t = 0; t < 2 * NKB; ++t)
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          const bf16x4 lo = lds_read_tr(vl + 16 * t * VSTR + 32 * db);
          const bf16x4 hi = lds_read_tr(vl + (16 * t + 8) * VSTR + 32 * db);
          const bf16x8 a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[t], oacc[db], 0, 0, 0);
        }
      // keep two MFMAs' worth of transposed V reads in flight
      __builtin_amdgcn_sched_group_barrier(0x100, 4, 1);
#pragma unroll
      for (int i = 0; i < (D / 32) * 2 * NKB - 2; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 1);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 1);
    }
    if (has_next) WAVEPP_STORE_TILE(buf ^ 1)
    __syncthreads();
  }
#undef WAVEPP_TILE_PAGES
#undef WAVEPP_LOAD_TILE
#undef WAVEPP_STORE_TILE

  // ---- epilogue: O = O^T / l, lse = ln(l) + m (natural log) ------------------------------------
  if (!row_ok) return;
  const float inv_l = l_run > 0.0f ? 1.0f / l_run : 0.0f;
  const float lse_v = l_run > 0.0f ? (m_run + __log2f(l_run)) * kLn2 : -INFINITY;
  if (it.part < 0) {
    __bf16* orow = out + (int64_t(rm.cu + tok) * Hq + head) * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        bf16x4 v;
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = static_cast<__bf16>(oacc[db][4 * u + k] * inv_l);
        *reinterpret_cast<bf16x4*>(orow + 32 * db + 8 * u + 4 * hf) = v;
      }
    if (lse_out && hf == 0) lse_out[int64_t(rm.cu + tok) * Hq + head] = lse_v;
  } else {
    float* orow = p.opart + int64_t(it.part + lrow) * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        f32x4 v;
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = oacc[db][4 * u + k] * inv_l;
        *reinterpret_cast<f32x4*>(orow + 32 * db + 8 * u + 4 * hf) = v;
      }
    if (hf == 0) p.lpart[it.part + lrow] = lse_v;
  }
}

// ---------------------------------------------------------------------------------------------
// Latent attention in absorbed form: every query head attends over one shared 576-wide latent per
// token (keys = the whole latent, values = its first 512 lanes).  Page size PAGE (16 or 64).
//
// One workgroup = 4 waves (one per SIMD) = 128 query rows; latent tiles of 64 keys.  Each staged
// 72 KiB tile serves 128 rows, so the L2 -> LDS traffic per FLOP is half that of 64-row items.
//   * Logits: wave w computes S^T for its own 32 rows (row block w) against both 32-key blocks of
//     the tile: 2 x 36 MFMAs sharing each Q fragment, with its 32 Q rows in registers.  The P.V
//     accumulators take all 256 AGPRs, so the logit MFMAs are inline assembly with VGPR
//     accumulators (mfma_v_pair).
//   * Softmax reference: fixed per row at the item's first tile (the row's two lanes hold its
//     maximum over the tile's 64 keys between them) and never moved, so the accumulators are never
//     rescaled.  If a later logit exceeds the reference by more than 2^64 the workgroup redoes its
//     key range with the exact row maxima (tracked per lane, combined at the end).
//   * Values: the bf16 probabilities, already in MFMA B-operand order, go through LDS; wave w
//     accumulates O for all 128 rows on value lanes [128w, 128w + 128), so each transposed V
//     fragment read from LDS feeds four MFMAs.
//   * The next latent tile is copied global -> LDS by the DMA path (global_load_lds, 16 bytes per
//     lane) into the other of two buffers; no registers stage it.  Its 18 instructions per wave go
//     one after every fourth logit MFMA: issued back to back they fill the vector-memory queue and
//     stall the wave for longer than the MFMAs they would otherwise overlap.  Each instruction's
//     source is a scalar page base plus a 32-bit lane offset rebuilt next to its use.
//     The two buffers are distinct LDS objects, and the current and next buffer pointers select
//     between them on the same condition, so the compiler can tell that the DMAs never touch the
//     buffer being read: the logit reads of the current buffer do not wait for the DMAs in flight
//     (the P.V reads are inline assembly, below).  The barrier between the probability writes and
//     the P.V reads only orders LDS accesses (the DMAs stay in flight); the barrier at the end of
//     a tile waits for them.  The page index of the tile after next is loaded a tile ahead.
//   * LDS: two 72 KiB tile buffers and 16 KiB of probabilities, the whole 160 KiB; after a pass the
//     probability buffer also carries the waves' overflow flags and the row sums.
//   * Layout of a tile in LDS: 64 rows of 72 16-byte chunks, unpadded; chunk c of row j is stored
//     at chunk position c ^ swz(j) of that row.  The swizzle puts the 16 rows read together by a
//     K fragment load, and the 4 rows x 4 chunks read together by a transposed V load, on distinct
//     banks.
// ---------------------------------------------------------------------------------------------
namespace mla {
constexpr int DQ = 576, DV = 512, KT = 64;
constexpr int CPR = DQ / 8;                  // 16-byte chunks per latent row (72)
constexpr int ROW_BYTES = DQ * 2;            // 1152
constexpr int TILE_BYTES = KT * ROW_BYTES;   // 73728
constexpr int NDMA = KT * CPR / 64 / 4;      // DMA instructions (64 lanes x 16 bytes) per wave per tile: 18
static_assert(NDMA * 4 * 64 == KT * CPR, "tile covered exactly by the DMA instructions");
constexpr int RPI = kMlaRowsPerItem;         // query rows per work item (32 per wave)
static_assert(RPI == 128 && kMlaKvTile == KT, "planner and kernel agree");
// chunk position of logical chunk c of row j: c ^ swz(j) (swz < 8 keeps it in c's aligned group of 8)
__device__ __forceinline__ uint32_t swz(uint32_t j) { return (((j >> 1) & 1u) << 2) | ((j >> 2) & 3u); }
}  // namespace mla

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) unsigned char lds_u8;
typedef __attribute__((address_space(3))) const bf16x8 lds_bf16x8;

// Barrier for LDS data only: this wave's LDS reads and writes have completed, then the workgroup
// meets.  Unlike __syncthreads() it does not wait for the wave's outstanding DMA loads into LDS.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0); vector-memory and export counts left unwaited
  asm volatile("s_barrier" ::: "memory");
}

// LDS reads of the latent kernel's P.V step, issued as inline assembly.  The compiler cannot tell
// that a transposed read (ds_read_b64_tr_b16) of the current tile misses the next tile's DMA into
// the other buffer, so with its own reads it would wait for the whole DMA (vmcnt(0)) before the
// first P.V fragment.  These reads are invisible to its wait tracking; the loop waits for each
// group of fragments itself with s_waitcnt lgkmcnt(0), tied to the group's values, after the next
// group has been issued.  lgkmcnt(0) also covers any scalar load in flight, so the wait is exact.
template <int OFF>
__device__ __forceinline__ bf16x8 lds_rd_b128(const lds_u8* p) {
  bf16x8 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(p), "i"(OFF) : "memory");
  return r;
}
template <int OFF>
__device__ __forceinline__ bf16x4 lds_rd_tr(const lds_u8* p) {
  bf16x4 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(p), "i"(OFF) : "memory");
  return r;
}
__device__ __forceinline__ void lds_wait4(bf16x8& a, bf16x8& b, bf16x8& c, bf16x8& d) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(b), "+v"(c), "+v"(d) :: "memory");
}
__device__ __forceinline__ void lds_wait_tr8(bf16x4 (&f)[8]) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]), "+v"(f[4]), "+v"(f[5]), "+v"(f[6]), "+v"(f[7])
               :: "memory");
}


// Logit MFMAs of the latent kernel, as inline assembly with their accumulators in VGPRs.  The P.V
// accumulators of the 128-row form fill all 256 AGPRs, and the compiler gives every MFMA of a
// function that uses AGPRs the AGPR form, so with the builtin the logit accumulators would push O
// out of its registers.  Hazards the compiler cannot see here are covered explicitly: two wait
// states before each pair (a VALU write of an operand), none between pairs of one chain (each
// accumulates into exactly its own registers), and 24 after the last pair before any other
// instruction reads or writes the results (mfma_v_drain).
__device__ __forceinline__ void mfma_v_pair0(f32x16& a0, f32x16& a1, const bf16x8& k0, const bf16x8& k1,
                                             const bf16x8& qv) {
  asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %2, %4, 0\n\tv_mfma_f32_32x32x16_bf16 %1, %3, %4, 0"
               : "=&v"(a0), "=&v"(a1) : "v"(k0), "v"(k1), "v"(qv));
}
__device__ __forceinline__ void mfma_v_pair(f32x16& a0, f32x16& a1, const bf16x8& k0, const bf16x8& k1,
                                            const bf16x8& qv) {
  asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %2, %4, %0\n\tv_mfma_f32_32x32x16_bf16 %1, %3, %4, %1"
               : "+v"(a0), "+v"(a1) : "v"(k0), "v"(k1), "v"(qv));
}
__device__ __forceinline__ void mfma_v_drain(f32x16& a0, f32x16& a1) {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(a0), "+v"(a1));
}

template <int PAGE>
__global__ __launch_bounds__(256, 1) void attn_mla_kernel(DevPlan p, const __bf16* __restrict__ q,
                                                          const __bf16* __restrict__ lat, __bf16* __restrict__ out,
                                                          float* __restrict__ lse_out) {
  using namespace mla;
  constexpr int PPT = (PAGE >= KT) ? 1 : KT / PAGE;   // pages per tile
  constexpr int NRB = RPI / 32;                       // row blocks (one per wave)
  __shared__ __attribute__((aligned(1024))) unsigned char lt0[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) unsigned char lt1[TILE_BYTES];
  // probabilities [row block][16-key step][lane]; after a pass the same bytes carry the workgroup's
  // flags and row sums
  __shared__ __attribute__((aligned(16))) bf16x8 pbuf[NRB][4][64];
  float* const xf = reinterpret_cast<float*>(&pbuf[0][0][0]);

  if (!meta_ok(p)) return;
  const WorkItem it = p.items[blockIdx.x];
  if (it.rows <= 0) return;
  const ReqMeta rm = p.reqs[it.req];
  const int Hq = p.num_q_heads;
  const int G = Hq;                     // a single latent head
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, col = lane & 31, hf = lane >> 5;
  const int rb = wave;
  const int n_valid = rm.prefix + rm.chunk;
  const int32_t* __restrict__ bt = p.bt + rm.bt_row;
  const int64_t page_stride = int64_t(PAGE) * DQ;

  // ---- this lane's logit row: row block rb; rows past it.rows repeat row 0 (never written) ------
  const int lrow = rb * 32 + col;
  const bool row_ok = lrow < it.rows;
  const int prow = it.row0 + (row_ok ? lrow : 0);
  const int tok = prow / G;
  const int limit = rm.prefix + tok;
  bf16x8 qf[DQ / 16];
  {
    const __bf16* qrow = q + (int64_t(rm.cu + tok) * Hq + (prow - tok * G)) * DQ + 8 * hf;
#pragma unroll
    for (int s = 0; s < DQ / 16; ++s) qf[s] = *reinterpret_cast<const bf16x8*>(qrow + 16 * s);
  }
  // smallest limit among the row block's lanes (lanes past it.rows use row 0's limit)
  const int blk_min_lim = rm.prefix + (it.row0 + ((rb * 32 + 32 <= it.rows) ? rb * 32 : 0)) / G;
  const float sl2 = p.softmax_scale * kLog2e;
  const int bound_base = min(limit, it.kv_end - 1) - 4 * hf;

  // ---- per-lane LDS byte offsets ---------------------------------------------------------------
  // K fragment of key block kb, step s = 4a + b: row 32kb + col, chunk 2s + hf
  //   -> kofs[b] + 36864 kb + 128a (the swizzle has period 16 in the row)
  int kofs[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) kofs[b] = col * ROW_BYTES + 16 * int((2u * b + hf) ^ swz(uint32_t(col)));
  // transposed V fragment of step t (16 keys), value block db (32 lanes of d), half lo/hi:
  //   rows 16t + 4hf + (lane & 15) / 4 (+8 for hi), d = 128 wave + 32 db + 16 g + 4 (lane & 3)
  //   -> (db even ? va : vb) + 128 (db >> 1) + 18432 t (+ dhi for hi)
  int va, vb, dhi;
  {
    const int g = (lane >> 4) & 1;
    const int j = 4 * hf + (lane & 15) / 4;
    const int fj = int(swz(uint32_t(j)));
    const int cf = (16 * wave + 2 * g + ((lane & 3) >> 1)) ^ fj;
    const int fb2 = (fj >> 2) & 1;
    const int x = j * ROW_BYTES + 16 * cf - 64 * fb2 + 8 * (lane & 1);
    va = x + 64 * fb2;
    vb = x + 64 * (1 - fb2);
    dhi = 8 * ROW_BYTES + (((cf >> 1) & 1) ? -32 : 32);
  }

  // ---- DMA of one latent tile into an LDS buffer ------------------------------------------------
  // Instruction i of wave w writes chunk positions P = 64 (w + 4i) + l (lane l) of the buffer; the
  // position holds logical chunk (P % 72) ^ swz(P / 72) of row P / 72, i.e. the tile's bytes at
  // 16 P + 16 d_i, where d_i = ((P % 8) ^ swz(P / 72)) - P % 8 lies in [-7, 7].  For whole tiles of
  // 64-token pages (the tile is one page) a lane keeps 16 P_0 and the 18 values 16 d_i packed in
  // bytes, so an instruction's source offset costs two ALU operations.  Other tiles (the request's
  // last, partial one, or 16-token pages) compute row and chunk directly; rows past the request's
  // last valid position copy that position's row (finite; the mask gives them zero weight), so
  // stale or NaN pool slots are never read.
  const int last_block = (n_valid - 1) / PAGE;
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t dma_o0 = 16u * uint32_t(64 * wave + lane);
  uint32_t dma_d[(NDMA + 3) / 4] = {};
#pragma unroll
  for (int i = 0; i < NDMA; ++i) {
    const uint32_t P = uint32_t(64 * (wave + 4 * i) + lane);
    const int q7 = int(P % CPR) & 7;
    const int d = ((q7 ^ int(swz(P / CPR))) - q7) * 16;
    dma_d[i / 4] |= (uint32_t(d) & 0xFFu) << (8 * (i % 4));
  }
  auto dma_tile = [&](lds_u8* buf, int tile) {
    const int kbase = tile * KT;
    if (PAGE >= KT && kbase + KT <= n_valid) {
      const int pg = __builtin_amdgcn_readfirstlane(bt[tile]);
      const char* tbase = reinterpret_cast<const char*>(lat + int64_t(pg) * page_stride);
#pragma unroll
      for (int i = 0; i < NDMA; ++i) {
        const int d = int(dma_d[i / 4] << (24 - 8 * (i % 4))) >> 24;
        __builtin_amdgcn_global_load_lds(tbase + (dma_o0 + 4096u * i + d), (lds_void*)(buf + 1024 * (wave_s + 4 * i)),
                                         16, 0, 0);
      }
      return;
    }
    const uint32_t jmax = uint32_t(n_valid - 1 - kbase);
    // this path runs once or twice per item: its per-lane indices are rebuilt here rather than hoisted
    // to the kernel start and kept (or spilled) for the whole item
    uint32_t lane_w = uint32_t(64 * wave + lane);
    asm volatile("" : "+v"(lane_w));
    int pg[PPT];
#pragma unroll
    for (int i = 0; i < PPT; ++i) pg[i] = bt[min(tile * (KT / PAGE) + i, last_block)];
#pragma unroll
    for (int i = 0; i < NDMA; ++i) {
      const uint32_t P = lane_w + 256u * i;
      const uint32_t j = P / CPR;
      const uint32_t c = (P - CPR * j) ^ swz(j);
      const uint32_t je = min(j, jmax);
      int page = pg[0];
#pragma unroll
      for (int u = 1; u < PPT; ++u) page = (je / PAGE == uint32_t(u)) ? pg[u] : page;
      __builtin_amdgcn_global_load_lds(lat + int64_t(page) * page_stride + ((je % PAGE) * DQ + 8 * c),
                                       (lds_void*)(buf + 1024 * (wave_s + 4 * i)), 16, 0, 0);
    }
  };

  f32x16 oacc[NRB][4];                  // [row block][value block]: O^T for value lanes 128 wave + 32 db
  float l_lane = 0.0f;                  // this lane's part of its row's sum (its half of every tile)
  float m_ref = -INFINITY;              // row reference (log2 units, scaled)
  float m_lane = -INFINITY;             // largest scaled logit this lane saw
  const int t_begin = it.kv_begin / KT;
  const int t_end = (it.kv_end + KT - 1) / KT;

  for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
    for (int r2 = 0; r2 < NRB; ++r2)
#pragma unroll
      for (int db = 0; db < 4; ++db) oacc[r2][db] = f32x16{};
    l_lane = 0.0f;
    dma_tile((lds_u8*)lt0, t_begin);
    int pg_next = (PAGE >= KT) ? bt[min(t_begin + 1, last_block)] : 0;   // made scalar at its use, a tile later
    __syncthreads();
    for (int tile = t_begin; tile < t_end; ++tile) {
      // both pointers select on the same condition: the compiler can tell that the DMAs into `nxt`
      // never touch `cur`, so the reads of `cur` do not wait for them
      const bool odd = (tile - t_begin) & 1;
      const lds_u8* cur = odd ? (const lds_u8*)lt1 : (const lds_u8*)lt0;
      lds_u8* nxt = odd ? (lds_u8*)lt0 : (lds_u8*)lt1;
      const bool set_ref = pass == 0 && tile == t_begin;
      // One tile: the next tile's DMA into `nxt`, logits of the wave's 32 rows against all 64 keys
      // from `cur`, probabilities to LDS, then O for all rows on the wave's value lanes.
      // whole next tiles of 64-token pages: the 18 DMA instructions go one per four logit MFMAs, so
      // the wave never stalls on a full vector-memory queue; the page index was loaded a tile ahead
      const bool dma_spread = PAGE >= KT && tile + 2 <= t_end && (tile + 2) * KT <= n_valid;
      const char* nbase = reinterpret_cast<const char*>(lat + int64_t(__builtin_amdgcn_readfirstlane(pg_next)) * page_stride);
      if (tile + 1 < t_end && !dma_spread) dma_tile(nxt, tile + 1);
      pg_next = bt[min(tile + 2, last_block)];
      // the DMA offsets are rebuilt next to each use (two ALU operations) instead of being held in
      // 18 registers across the loop
      asm volatile("" : "+v"(dma_d[0]), "+v"(dma_d[1]), "+v"(dma_d[2]), "+v"(dma_d[3]), "+v"(dma_d[4]));
      const int kbase = tile * KT;
      // S^T of both key blocks: 2 x 36 MFMAs sharing each Q fragment; K fragments read KPF steps
      // ahead, in source order, so the reads stay in flight behind the MFMAs (three steps measured
      // 1.5 % faster on cfg5 than two; four spill)
      f32x16 sacc[2];
      {
        constexpr int KPF = 3;
        bf16x8 kbuf[2][KPF];
  #pragma unroll
        for (int i = 0; i < KPF; ++i) {
          kbuf[0][i] = *reinterpret_cast<lds_bf16x8*>(cur + kofs[i & 3] + 128 * (i >> 2));
          kbuf[1][i] = *reinterpret_cast<lds_bf16x8*>(cur + kofs[i & 3] + 128 * (i >> 2) + 32 * ROW_BYTES);
        }
  #pragma unroll
        for (int s = 0; s < DQ / 16; ++s) {
          const bf16x8 k0 = kbuf[0][s % KPF], k1 = kbuf[1][s % KPF];
          if (s + KPF < DQ / 16) {
            const int n = s + KPF;
            kbuf[0][s % KPF] = *reinterpret_cast<lds_bf16x8*>(cur + kofs[n & 3] + 128 * (n >> 2));
            kbuf[1][s % KPF] = *reinterpret_cast<lds_bf16x8*>(cur + kofs[n & 3] + 128 * (n >> 2) + 32 * ROW_BYTES);
          }
          if (dma_spread && (s & 1) == 0) {
            const int i = s >> 1;
            const int d = int(dma_d[i / 4] << (24 - 8 * (i % 4))) >> 24;
            __builtin_amdgcn_global_load_lds(nbase + (dma_o0 + 4096u * i + d), (lds_void*)(nxt + 1024 * (wave_s + 4 * i)),
                                             16, 0, 0);
          }
          // the scheduler would otherwise sink each read down to its MFMA (one read in flight)
          __builtin_amdgcn_sched_barrier(0);
          if (s == 0) mfma_v_pair0(sacc[0], sacc[1], k0, k1, qf[s]);
          else mfma_v_pair(sacc[0], sacc[1], k0, k1, qf[s]);
        }
        mfma_v_drain(sacc[0], sacc[1]);
      }
      // the first P.V step's transposed V fragments do not depend on the probabilities: read them now,
      // so that they land during the softmax
      const lds_u8* pva = cur + va;
      const lds_u8* pvb = cur + vb;
      const lds_u8* pha = cur + va + dhi;
      const lds_u8* phb = cur + vb + dhi;
      bf16x4 vraw[8];
      auto issue_v = [&](auto T, bf16x4 (&vr)[8]) {
        constexpr int o = 18432 * decltype(T)::value;
        vr[0] = lds_rd_tr<o>(pva);
        vr[1] = lds_rd_tr<o>(pha);
        vr[2] = lds_rd_tr<o>(pvb);
        vr[3] = lds_rd_tr<o>(phb);
        vr[4] = lds_rd_tr<o + 128>(pva);
        vr[5] = lds_rd_tr<o + 128>(pha);
        vr[6] = lds_rd_tr<o + 128>(pvb);
        vr[7] = lds_rd_tr<o + 128>(phb);
      };
      issue_v(std::integral_constant<int, 0>{}, vraw);
      // element r of sacc[kb] holds key kbase + 32 kb + 8 (r / 4) + 4 hf + (r % 4)
      float mx = -INFINITY;
  #pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        if ((kbase + 32 * kb + 31 > blk_min_lim) || (kbase + 32 * kb + 32 > it.kv_end)) {
          const int bound = bound_base - kbase - 32 * kb;
  #pragma unroll
          for (int r = 0; r < 16; ++r)
            if (8 * (r >> 2) + (r & 3) > bound) sacc[kb][r] = -INFINITY;
        }
  #pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kb][r]);
      }
      mx *= sl2;
      m_lane = fmaxf(m_lane, mx);
      // the item's first tile in the first pass (uniform over the workgroup): the reference is the
      // row maximum over the tile's 64 keys, which the row's two lanes hold between them; -inf means
      // the row sees no key of the item's range (its visible keys are a prefix of the range), so it
      // never needs one
      if (set_ref) m_ref = halves_max(mx);
      const float m_use = (m_ref == -INFINITY) ? 0.0f : m_ref;
  #pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        bf16x8 pb[2];
  #pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float e = fast_exp2(fmaf(sacc[kb][r], sl2, -m_use));
          l_lane += e;
          pb[r >> 3][r & 7] = static_cast<__bf16>(e);
        }
        pbuf[rb][2 * kb][lane] = pb[0];
        pbuf[rb][2 * kb + 1][lane] = pb[1];
      }
      lds_barrier();
      // O^T[d][row] += V^T[d][key] P^T[key][row]; step t covers keys 16t + 8 (e / 4) + 4 hf + (e % 4).
      // Step t + 1's fragments (four probability fragments, eight transposed V halves) are read while
      // the sixteen MFMAs of step t run; a fragment's halves are joined only after the wait for them.
      {
        const lds_u8* pp0 = (const lds_u8*)(&pbuf[0][0][lane]);
        auto issue_p = [&](auto T, bf16x8 (&pd)[NRB]) {
          constexpr int t = decltype(T)::value;
          pd[0] = lds_rd_b128<1024 * t>(pp0);
          pd[1] = lds_rd_b128<4096 + 1024 * t>(pp0);
          pd[2] = lds_rd_b128<8192 + 1024 * t>(pp0);
          pd[3] = lds_rd_b128<12288 + 1024 * t>(pp0);
        };
        auto join = [&](bf16x4 (&vr)[8], bf16x8 (&vd)[4]) {
#pragma unroll
          for (int db = 0; db < 4; ++db) vd[db] = __builtin_shufflevector(vr[2 * db], vr[2 * db + 1], 0, 1, 2, 3, 4, 5, 6, 7);
        };
        bf16x8 pa[NRB], pn[NRB], va4[4];
        bf16x4 vn[8];
        issue_p(std::integral_constant<int, 0>{}, pa);
        lds_wait_tr8(vraw);   // (landed before the barrier: this ties the values to the wait)
        lds_wait4(pa[0], pa[1], pa[2], pa[3]);
        join(vraw, va4);
        auto step = [&](auto T) {
          constexpr int t = decltype(T)::value;
          if constexpr (t + 1 < 4) {
            issue_p(std::integral_constant<int, t + 1>{}, pn);
            issue_v(std::integral_constant<int, t + 1>{}, vn);
          }
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int db = 0; db < 4; ++db)
#pragma unroll
            for (int r2 = 0; r2 < NRB; ++r2)
              oacc[r2][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va4[db], pa[r2], oacc[r2][db], 0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
          if constexpr (t + 1 < 4) {
            lds_wait_tr8(vn);
            asm volatile("" : "+v"(pn[0]), "+v"(pn[1]), "+v"(pn[2]), "+v"(pn[3]));
#pragma unroll
            for (int r2 = 0; r2 < NRB; ++r2) pa[r2] = pn[r2];
            join(vn, va4);
          }
        };
        step(std::integral_constant<int, 0>{}); step(std::integral_constant<int, 1>{});
        step(std::integral_constant<int, 2>{}); step(std::integral_constant<int, 3>{});
      }
      __syncthreads();   // the next tile's DMA has landed; this tile's reads are done
    }
    // A reference exceeded by more than 2^64 (log2 units): redo the range with the exact maxima.
    // The row's two lanes hold its maximum between them; the waves' verdicts meet in LDS (the
    // probability buffer is idle after the loop's last barrier).
    const float m_row = halves_max(m_lane);
    const bool exceeded = (m_ref != -INFINITY) && (m_row > m_ref + 64.0f);
    const bool wave_any = __builtin_amdgcn_ballot_w64(exceeded) != 0;
    if (lane == 0) xf[wave] = wave_any ? 1.0f : 0.0f;
    __syncthreads();
    bool any = false;
#pragma unroll
    for (int w = 0; w < NRB; ++w) any = any || (xf[w] != 0.0f);
    __syncthreads();   // the flags are read before the next pass writes probabilities
    if (pass == 1 || !any) break;
    m_ref = m_row;
    m_lane = -INFINITY;
  }

  // ---- epilogue: row sums through LDS; every wave normalizes its value lanes of all rows ----------
  const float l_row = halves_sum(l_lane);
  if (hf == 0) xf[32 * rb + col] = l_row;
  __syncthreads();
  if (hf == 0 && row_ok) {
    const float m_use = (m_ref == -INFINITY) ? 0.0f : m_ref;
    const float lse_v = l_row > 0.0f ? (m_use + __log2f(l_row)) * kLn2 : -INFINITY;
    if (it.part < 0) {
      if (lse_out) lse_out[int64_t(rm.cu + tok) * Hq + (prow - tok * G)] = lse_v;
    } else {
      p.lpart[it.part + lrow] = lse_v;
    }
  }
#pragma unroll
  for (int r2 = 0; r2 < NRB; ++r2) {
    const int r_local = 32 * r2 + col;
    if (r_local >= it.rows) continue;
    const float l = xf[r_local];
    const float inv_l = l > 0.0f ? 1.0f / l : 0.0f;
    const int pr = it.row0 + r_local;
    const int tk = pr / G;
    const int hd = pr - tk * G;
    if (it.part < 0) {
      __bf16* orow = out + (int64_t(rm.cu + tk) * Hq + hd) * DV + 128 * wave;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          bf16x4 v;
#pragma unroll
          for (int k = 0; k < 4; ++k) v[k] = static_cast<__bf16>(oacc[r2][db][4 * u + k] * inv_l);
          *reinterpret_cast<bf16x4*>(orow + 32 * db + 8 * u + 4 * hf) = v;
        }
    } else {
      float* orow = p.opart + int64_t(it.part + r_local) * DV + 128 * wave;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          f32x4 v;
#pragma unroll
          for (int k = 0; k < 4; ++k) v[k] = oacc[r2][db][4 * u + k] * inv_l;
          *reinterpret_cast<f32x4*>(orow + 32 * db + 8 * u + 4 * hf) = v;
        }
    }
  }
}

// ---------------------------------------------------------------------------------------------
// Metadata upload: the plan's bytes, read straight from the pinned (coherent, device-mapped)
// staging buffer and written into the workspace.  A kernel on the launch stream keeps the upload
// in the compute queue, so the append and attention kernels behind it start without waiting for
// a DMA engine's completion signal.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void upload_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                     int64_t n16) {
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n16; i += int64_t(gridDim.x) * 256) dst[i] = src[i];
}

// ---------------------------------------------------------------------------------------------
// Merge of key-range splits: o = sum_s w_s o_s / sum_s w_s with w_s = exp(lse_s - max lse),
// lse = max + ln sum_s w_s.  Splits are combined in index order, so results are deterministic.
// ---------------------------------------------------------------------------------------------
template <int DV>
__global__ __launch_bounds__(256) void merge_kernel(DevPlan p, __bf16* __restrict__ out, float* __restrict__ lse_out) {
  // workgroup (x = merge item, y = row group) handles RPB rows; one thread per (row, 4 value lanes)
  constexpr int C4 = DV / 4;
  constexpr int RPB = 256 / C4;
  if (!meta_ok(p)) return;
  const MergeItem mi = p.merges[blockIdx.x];
  const int lrow = blockIdx.y * RPB + threadIdx.x / C4;
  const int c4 = threadIdx.x % C4;
  if (lrow >= mi.rows) return;
  const ReqMeta rm = p.reqs[mi.req];
  const int Hq = p.num_q_heads, G = Hq / p.num_kv_heads;
  // The accumulation order is s = 0, 1, ..., nsplit - 1 (deterministic).  A split that saw no key
  // has lse = -inf and an all-zero partial row, which gets weight 0.  Up to SB splits, every LSE and
  // partial is loaded at once (one memory round trip); beyond that, two passes read four splits at
  // a time.  Both paths do the same arithmetic in the same order.
  constexpr int SB = 16;
  const int ns = mi.nsplit;
  const float* __restrict__ lp = p.lpart + mi.part + lrow;
  const float* __restrict__ op = p.opart + (int64_t(mi.part) + lrow) * DV + 4 * c4;
  const int64_t ostep = int64_t(mi.rows) * DV;
  float mx = -INFINITY;
  f32x4 acc = f32x4{};
  float wsum = 0.0f;
  if (ns <= SB) {
    float l[SB];
    f32x4 v[SB];
#pragma unroll
    for (int u = 0; u < SB; ++u) {
      l[u] = u < ns ? lp[u * mi.rows] : -INFINITY;
      v[u] = u < ns ? *reinterpret_cast<const f32x4*>(op + u * ostep) : f32x4{};
    }
#pragma unroll
    for (int u = 0; u < SB; ++u) mx = fmaxf(mx, l[u]);
#pragma unroll
    for (int u = 0; u < SB; ++u) {
      if (u < ns) {
        const float w = (l[u] == -INFINITY) ? 0.0f : fast_exp2((l[u] - mx) * kLog2e);
        acc += w * v[u];
        wsum += w;
      }
    }
  } else {
    {
      int s = 0;
      for (; s + 4 <= ns; s += 4) {
        float l[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) l[u] = lp[(s + u) * mi.rows];
#pragma unroll
        for (int u = 0; u < 4; ++u) mx = fmaxf(mx, l[u]);
      }
      for (; s < ns; ++s) mx = fmaxf(mx, lp[s * mi.rows]);
    }
    {
      int s = 0;
      for (; s + 4 <= ns; s += 4) {
        float l[4];
        f32x4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          l[u] = lp[(s + u) * mi.rows];
          v[u] = *reinterpret_cast<const f32x4*>(op + (s + u) * ostep);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float w = (l[u] == -INFINITY) ? 0.0f : fast_exp2((l[u] - mx) * kLog2e);
          acc += w * v[u];
          wsum += w;
        }
      }
      for (; s < ns; ++s) {
        const float l = lp[s * mi.rows];
        const float w = (l == -INFINITY) ? 0.0f : fast_exp2((l - mx) * kLog2e);
        acc += w * *reinterpret_cast<const f32x4*>(op + s * ostep);
        wsum += w;
      }
    }
  }
  const float inv = 1.0f / wsum;
  const int row = mi.row0 + lrow;
  const int tok = row / G;
  const int head = mi.kv_head * G + (row - tok * G);
  bf16x4 o;
#pragma unroll
  for (int k = 0; k < 4; ++k) o[k] = static_cast<__bf16>(acc[k] * inv);
  const int64_t orow = int64_t(rm.cu + tok) * Hq + head;
  *reinterpret_cast<bf16x4*>(out + orow * DV + 4 * c4) = o;
  if (lse_out && c4 == 0) lse_out[orow] = mx + __logf(wsum);
}

// ---------------------------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------------------------
hipError_t launch_append(const DevPlan& p, const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                         hipStream_t stream) {
  const int dk = p.head_dim_qk, dv = p.kv_shared ? 0 : p.head_dim_v;
  if (p.total_tokens == 0) return hipSuccess;
  const int64_t blocks = (p.total_tokens + kAppendTokens - 1) / kAppendTokens;
  if (blocks > INT32_MAX) return hipErrorInvalidValue;
  const int per_tok = p.num_kv_heads * ((dk + dv) / 8);
  const int threads = std::min(256, (per_tok + 63) / 64 * 64);
  auto kn = static_cast<const uint4*>(k_new);
  auto vn = static_cast<const uint4*>(v_new);
  auto kp = static_cast<uint4*>(k_pool);
  auto vp = static_cast<uint4*>(v_pool);
  if (dk == 64 && dv == 64)
    hipLaunchKernelGGL((append_kernel<64, 64>), dim3(blocks), dim3(threads), 0, stream, p, kn, vn, kp, vp);
  else if (dk == 128 && dv == 128)
    hipLaunchKernelGGL((append_kernel<128, 128>), dim3(blocks), dim3(threads), 0, stream, p, kn, vn, kp, vp);
  else if (dk == 576 && dv == 0)
    hipLaunchKernelGGL((append_kernel<576, 0>), dim3(blocks), dim3(threads), 0, stream, p, kn, vn, kp, vp);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attention(const DevPlan& p, const void* q, const void* k_pool, const void* v_pool, void* out,
                            float* lse, hipStream_t stream) {
  if (p.num_items == 0) return hipSuccess;
  auto qq = static_cast<const __bf16*>(q);
  auto kp = static_cast<const __bf16*>(k_pool);
  auto vp = static_cast<const __bf16*>(v_pool);
  auto oo = static_cast<__bf16*>(out);
  const dim3 grid(p.num_items), block(256);
  if (p.kv_shared) {
    if (p.head_dim_qk != 576 || p.head_dim_v != 512) return hipErrorInvalidValue;
    if (p.page_size == 64)
      hipLaunchKernelGGL((attn_mla_kernel<64>), grid, block, 0, stream, p, qq, kp, oo, lse);
    else if (p.page_size == 16)
      hipLaunchKernelGGL((attn_mla_kernel<16>), grid, block, 0, stream, p, qq, kp, oo, lse);
    else
      return hipErrorInvalidValue;
    return hipGetLastError();
  }
  const bool w8 = p.rows_per_item == 256;
  if (!w8 && p.rows_per_item != 128) return hipErrorInvalidValue;
  const dim3 block_g(w8 ? 512 : 256);
#define WAVEPP_GQA(D_, P_)                                                                                 \
  if (w8) hipLaunchKernelGGL((attn_gqa_kernel<D_, P_, 8>), grid, block_g, 0, stream, p, qq, kp, vp, oo, lse); \
  else hipLaunchKernelGGL((attn_gqa_kernel<D_, P_, 4>), grid, block_g, 0, stream, p, qq, kp, vp, oo, lse);
  if (p.head_dim_qk == 128 && p.page_size == 64) {
    WAVEPP_GQA(128, 64)
  } else if (p.head_dim_qk == 128 && p.page_size == 16) {
    WAVEPP_GQA(128, 16)
  } else if (p.head_dim_qk == 64 && p.page_size == 64) {
    WAVEPP_GQA(64, 64)
  } else if (p.head_dim_qk == 64 && p.page_size == 16) {
    WAVEPP_GQA(64, 16)
  } else {
    return hipErrorInvalidValue;
  }
#undef WAVEPP_GQA
  return hipGetLastError();
}

hipError_t launch_upload(const void* src, void* dst, size_t bytes, hipStream_t stream) {
  if (bytes == 0) return hipSuccess;
  // metadata blobs are built from 16-byte-aligned records
  if (bytes % 16 || reinterpret_cast<uintptr_t>(src) % 16 || reinterpret_cast<uintptr_t>(dst) % 16)
    return hipErrorInvalidValue;
  const int64_t n16 = int64_t(bytes / 16);
  const int64_t blocks = std::min<int64_t>((n16 + 255) / 256, 1024);
  hipLaunchKernelGGL(upload_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream, static_cast<const u32x4*>(src),
                     static_cast<u32x4*>(dst), n16);
  return hipGetLastError();
}

hipError_t launch_merge(const DevPlan& p, void* out, float* lse, hipStream_t stream) {
  if (p.num_merge == 0) return hipSuccess;
  auto oo = static_cast<__bf16*>(out);
  const int c4 = p.head_dim_v / 4;
  const int rpb = 256 / c4;
  const dim3 grid(p.num_merge, (p.rows_per_item + rpb - 1) / rpb), block(256);
  if (p.head_dim_v == 128)
    hipLaunchKernelGGL((merge_kernel<128>), grid, block, 0, stream, p, oo, lse);
  else if (p.head_dim_v == 64)
    hipLaunchKernelGGL((merge_kernel<64>), grid, block, 0, stream, p, oo, lse);
  else if (p.head_dim_v == 512)
    hipLaunchKernelGGL((merge_kernel<512>), grid, block, 0, stream, p, oo, lse);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------------
// Scratch of the allocation-free entry point (wavepp_attn_chunked_prefill_noalloc): the plan's
// metadata and its split partials live in this static device array instead of a caller workspace.
// Each GPU the library runs on holds its own copy until the process ends.  In host code the name
// `scratch` is only a host-side stand-in: its device address is taken once per device with
// hipGetSymbolAddress and only that address is handed to kernels and copies.
// ---------------------------------------------------------------------------------------------
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));   // the current device's copy of the array
    if (e != hipSuccess) return e;
    if (!p || reinterpret_cast<uintptr_t>(p) % 256) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace wavepp
