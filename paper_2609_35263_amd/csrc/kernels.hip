// gfx950 (CDNA4) kernels of libwavepp_attn: K/V append into reserved pages, chunked-prefill
// attention over paged K/V with bf16 MFMA, and the merge of key-range splits.
//
// Attention layout (one workgroup = 4 waves = one work item of up to 128 query rows):
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
//   * K/V tiles of 64 keys are gathered from the pages named by the block table with 16-byte
//     loads (one page's head slice is contiguous), double-buffered in LDS: the next tile's global
//     loads are issued before the current tile's MFMAs and written to the other buffer after.
//   * Online softmax in fp32 (exp2 with the log2(e) factor folded into the scale); masking is by
//     selection, and K/V rows past the request's last valid position are never loaded (their
//     addresses are clamped to the last valid row), so stale or NaN pool slots cannot leak into
//     the output.
#include <hip/hip_runtime.h>

#include "internal.h"

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
// One thread moves one 16-byte chunk; the flat index runs over (token, kv head, chunk).
// ---------------------------------------------------------------------------------------------
template <int DK, int DV>
__global__ __launch_bounds__(256) void append_kernel(DevPlan p, const uint4* __restrict__ k_new,
                                                     const uint4* __restrict__ v_new, uint4* __restrict__ k_pool,
                                                     uint4* __restrict__ v_pool) {
  if (!meta_ok(p)) return;
  constexpr int KC = DK / 8, VC = DV / 8, UC = KC + VC;
  const int Hkv = p.num_kv_heads;
  const int64_t units = p.total_tokens * Hkv * UC;
  const int B = p.page_size;
  for (int64_t u = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; u < units; u += int64_t(gridDim.x) * blockDim.x) {
    const int64_t per_tok = int64_t(Hkv) * UC;
    const int t = int(u / per_tok);
    const int rem = int(u - int64_t(t) * per_tok);
    const int h = rem / UC;
    const int c = rem - h * UC;
    // request holding token t: the last r with cu_r <= t (idle lanes share cu with the next one)
    int lo = 0, hi = p.num_requests - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (p.reqs[mid].cu <= t) lo = mid; else hi = mid - 1;
    }
    const ReqMeta rm = p.reqs[lo];
    const int pos = rm.prefix + (t - rm.cu);
    const int64_t page = p.bt[rm.bt_row + pos / B];
    const int slot = pos % B;
    if (c < KC) {
      k_pool[((page * Hkv + h) * B + slot) * KC + c] = k_new[(int64_t(t) * Hkv + h) * KC + c];
    } else {
      const int cv = c - KC;
      v_pool[((page * Hkv + h) * B + slot) * VC + cv] = v_new[(int64_t(t) * Hkv + h) * VC + cv];
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

template <int D, int PAGE>
__global__ __launch_bounds__(256, 2) void attn_gqa_kernel(DevPlan p, const __bf16* __restrict__ q,
                                                          const __bf16* __restrict__ kpool,
                                                          const __bf16* __restrict__ vpool, __bf16* __restrict__ out,
                                                          float* __restrict__ lse_out) {
  constexpr int KT = kKvTile;          // 64 keys per tile
  constexpr int KSTR = D + 8;          // K rows in LDS: 16-byte reads of 8 rows land on distinct banks
  constexpr int VSTR = D + 16;         // V rows in LDS: transposed reads of 4 rows x 32 bytes on distinct banks
  constexpr int CH = D / 8;            // 16-byte chunks per key row
  constexpr int LOADS = KT * CH / 256; // chunks per thread per tile, for K and for V alike
  constexpr int PPT = (PAGE >= KT) ? 1 : KT / PAGE;   // pages touched by one tile
  static_assert(LOADS * 256 == KT * CH, "tile covered exactly");
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
  // Thread tid moves 16-byte chunks c = tid + 256 i of both the K and the V tile: key c / CH, chunk
  // c % CH; consecutive threads read consecutive 16 bytes of a page's contiguous head slice.  The
  // physical pages of a tile are looked up one tile ahead (uniform across the workgroup, hence
  // scalar loads) and the loads of tile t+1 are issued before the MFMAs of tile t.  In the last
  // tile of a request, key positions past its last valid slot are clamped to that slot: those rows
  // are finite copies that the mask gives zero weight, so stale or NaN pool slots are never read.
  const int last_block = (n_valid - 1) / PAGE;
  int ckey[LOADS];
  uint32_t coff[LOADS];
#pragma unroll
  for (int i = 0; i < LOADS; ++i) {
    const int c = tid + 256 * i;
    ckey[i] = c / CH;
    coff[i] = uint32_t((c % CH) * 8);
  }
  u32x4 kreg[LOADS], vreg[LOADS];
  int pg_nxt[PPT];

#define WAVEPP_TILE_PAGES(tile_, pg_)                                                                     \
  _Pragma("unroll") for (int i_ = 0; i_ < PPT; ++i_) pg_[i_] = bt[min((tile_) * (KT / PAGE) + i_, last_block)];

#define WAVEPP_LOAD_TILE(tile_, pg_)                                                                      \
  {                                                                                                       \
    const int kbase_ = (tile_) * KT;                                                                      \
    const bool full_ = kbase_ + KT <= n_valid;                                                            \
    _Pragma("unroll") for (int i_ = 0; i_ < LOADS; ++i_) {                                                \
      const int j_ = full_ ? kbase_ + ckey[i_] : min(kbase_ + ckey[i_], n_valid - 1);                     \
      const int sub_ = (j_ - kbase_) / PAGE;                                                              \
      int page_ = pg_[0];                                                                                 \
      _Pragma("unroll") for (int q_ = 1; q_ < PPT; ++q_) page_ = (sub_ == q_) ? pg_[q_] : page_;          \
      const uint32_t off_ = uint32_t(j_ % PAGE) * D + coff[i_];                                           \
      kreg[i_] = *reinterpret_cast<const u32x4*>(kpool_h + int64_t(page_) * page_stride + off_);         \
      vreg[i_] = *reinterpret_cast<const u32x4*>(vpool_h + int64_t(page_) * page_stride + off_);         \
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
      // S^T[key][row] for the 64 keys of the tile, as two 32-key blocks
      f32x16 sacc[2] = {f32x16{}, f32x16{}};
      const __bf16* kl = &ks[buf][k_lane];
#pragma unroll
      for (int s = 0; s < D / 16; ++s)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          const bf16x8 kf = *reinterpret_cast<const bf16x8*>(kl + 32 * kb * KSTR + 16 * s);
          sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], sacc[kb], 0, 0, 0);
        }
      // keep four K fragment reads in flight ahead of the MFMAs that consume them
      __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
      for (int i = 0; i < D / 8 - 4; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
      // accumulator element r of block kb holds key 32*kb + 8*(r/4) + 4*hf + (r%4)
      const bool need_mask = (kbase + KT - 1 > wave_min_lim) || (kbase + KT > it.kv_end);
      if (need_mask) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = kbase + 32 * kb + 8 * (r >> 2) + 4 * hf + (r & 3);
            if (key > limit || key >= it.kv_end) sacc[kb][r] = -INFINITY;
          }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
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
      bf16x8 pb[4];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
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
      for (int t = 0; t < 4; ++t)
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
      for (int i = 0; i < D / 8 - 2; ++i) {
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
// Merge of key-range splits: o = sum_s w_s o_s / sum_s w_s with w_s = exp(lse_s - max lse),
// lse = max + ln sum_s w_s.  Splits are combined in index order, so results are deterministic.
// ---------------------------------------------------------------------------------------------
template <int DV>
__global__ __launch_bounds__(256) void merge_kernel(DevPlan p, __bf16* __restrict__ out, float* __restrict__ lse_out) {
  if (!meta_ok(p)) return;
  const MergeItem mi = p.merges[blockIdx.x];
  const ReqMeta rm = p.reqs[mi.req];
  const int Hq = p.num_q_heads, G = Hq / p.num_kv_heads;
  constexpr int C4 = DV / 4;
  for (int idx = threadIdx.x; idx < mi.rows * C4; idx += blockDim.x) {
    const int lrow = idx / C4, c4 = idx - lrow * C4;
    float mx = -INFINITY;
    for (int s = 0; s < mi.nsplit; ++s) mx = fmaxf(mx, p.lpart[mi.part + s * mi.rows + lrow]);
    f32x4 acc = f32x4{};
    float wsum = 0.0f;
    for (int s = 0; s < mi.nsplit; ++s) {
      const int prow = mi.part + s * mi.rows + lrow;
      const float l = p.lpart[prow];
      const float w = (l == -INFINITY) ? 0.0f : fast_exp2((l - mx) * kLog2e);
      if (w != 0.0f) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(p.opart + int64_t(prow) * DV + 4 * c4);
        acc += w * v;
      }
      wsum += w;
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
}

// ---------------------------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------------------------
hipError_t launch_append(const DevPlan& p, const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                         hipStream_t stream) {
  const int dk = p.head_dim_qk, dv = p.kv_shared ? 0 : p.head_dim_v;
  const int64_t units = p.total_tokens * p.num_kv_heads * ((dk + dv) / 8);
  if (units == 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((units + 255) / 256, 65536);
  auto kn = static_cast<const uint4*>(k_new);
  auto vn = static_cast<const uint4*>(v_new);
  auto kp = static_cast<uint4*>(k_pool);
  auto vp = static_cast<uint4*>(v_pool);
  if (dk == 64 && dv == 64)
    hipLaunchKernelGGL((append_kernel<64, 64>), dim3(blocks), dim3(256), 0, stream, p, kn, vn, kp, vp);
  else if (dk == 128 && dv == 128)
    hipLaunchKernelGGL((append_kernel<128, 128>), dim3(blocks), dim3(256), 0, stream, p, kn, vn, kp, vp);
  else if (dk == 576 && dv == 0)
    hipLaunchKernelGGL((append_kernel<576, 0>), dim3(blocks), dim3(256), 0, stream, p, kn, vn, kp, vp);
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
  if (p.kv_shared) return hipErrorInvalidValue;
  if (p.head_dim_qk == 128 && p.page_size == 64)
    hipLaunchKernelGGL((attn_gqa_kernel<128, 64>), grid, block, 0, stream, p, qq, kp, vp, oo, lse);
  else if (p.head_dim_qk == 128 && p.page_size == 16)
    hipLaunchKernelGGL((attn_gqa_kernel<128, 16>), grid, block, 0, stream, p, qq, kp, vp, oo, lse);
  else if (p.head_dim_qk == 64 && p.page_size == 64)
    hipLaunchKernelGGL((attn_gqa_kernel<64, 64>), grid, block, 0, stream, p, qq, kp, vp, oo, lse);
  else if (p.head_dim_qk == 64 && p.page_size == 16)
    hipLaunchKernelGGL((attn_gqa_kernel<64, 16>), grid, block, 0, stream, p, qq, kp, vp, oo, lse);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_merge(const DevPlan& p, void* out, float* lse, hipStream_t stream) {
  if (p.num_merge == 0) return hipSuccess;
  auto oo = static_cast<__bf16*>(out);
  const dim3 grid(p.num_merge), block(256);
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

}  // namespace wavepp
