// gfx950 (CDNA4) kernel of libwavepp_attn: chunked prefill of a KDA (gated delta-rule) layer that
// resumes from a recurrent-state snapshot and leaves the snapshot at the chunk boundary.
//
// Per head, with per-channel decay alpha_t, write strength beta_t, key k_t, value v_t, query q_t
// (Preliminaries, "Transformer Architectures", Eq. 2-3):
//   S_t = (I - beta_t k_t k_t^T) Diag(alpha_t) S_{t-1} + beta_t k_t v_t^T,   o_t = S_t^T q_t.
//
// Chunkwise form.  Tokens are processed in blocks of C = 64.  Inside a block, with S0 the state
// before it and gamma_t = alpha_1 * ... * alpha_t (per channel, running product from the block
// start), write the state change of token t as k_t u_t^T.  Unrolling the recurrence gives
//   u_t = beta_t (v_t - S0^T (gamma_t * k_t) - sum_{s<t} u_s <k_s / gamma_s, gamma_t * k_t>),
// i.e. (I + A) U = Diag(beta) (V - K~ S0) with K~ = gamma * K and the strictly lower-triangular
// A[t][s] = beta_t <gamma_t * k_t, k_s / gamma_s>.  With T = (I + A)^-1 and R = Diag(beta)(V - K~ S0):
//   U = T R,
//   O = Q~ S0 + P U,              Q~ = gamma * Q,  P[t][s] = <gamma_t * q_t, k_s / gamma_s> (s <= t),
//   S_C = Diag(gamma_C) S0 + Kbar^T U,   Kbar_s = k_s * gamma_C / gamma_s.
// Every product of 64-token blocks with the 128 x 128 state is a bf16 MFMA contraction with fp32
// accumulation; the state itself stays in fp32 accumulators for the whole chunk.
//
// Range.  The factorization gamma_t / gamma_s = gamma_t * (1 / gamma_s) is used for a channel only
// when its block decay gamma_C is at least 2^-96, so every factor stays a normal number.  Kbar is
// built from products of the later decays (gamma_C / gamma_s without a division) and
// 1 / gamma_s = (gamma_C / gamma_s) / gamma_C, one reciprocal per channel and block.  A
// channel that decays more within one block (including alpha = 0) is "slow": it contributes to A
// and P through an exact pairwise term exp2(G_t - G_s) in log2 space instead, and its Kbar uses
// exp2(G_C - G_s).
//
// Workgroup = one (request, head), 4 waves.  Wave w owns state columns [32w, 32w + 32) as four
// 32 x 32 fp32 accumulator tiles.  The accumulator layout of v_mfma_f32_32x32x16_bf16 (lane = column,
// 16 rows per lane) is reused directly as the B operand of the next contraction: the eight rows a lane
// holds for one MFMA are its contraction slots, and the A operand is read from LDS in that same
// (permuted) order.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace wavepp {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kC = kKdaBlock;       // tokens per block
constexpr int kD = kKdaDim;         // d_k = d_v
// LDS row strides.  The LDS has 64 banks of 4 bytes.  A permuted A-operand read (lds_a_perm) has the
// 32 lanes of a half-wave read 8 bytes each from 32 consecutive rows: with a row stride that is an odd
// multiple of 8 bytes modulo 256 those land on 32 distinct bank pairs.  Arrays read that way keep
// rows only 8-byte aligned and are accessed 8 bytes at a time.
constexpr int RS = kD + 8;          // bf16 row stride of K_R and of the staged output (16-byte accesses)
constexpr int QS = kD + 4;          // bf16 row stride of Q~ and K~: 264 B
constexpr int VS = kD + 32;         // bf16 row stride of V: 320 B, so that the 4 rows x 64 B of a
                                    // transposing read cover the 64 banks once
constexpr int CS = kC + 4;          // bf16 row stride of [channel][t] arrays and of P, T [t][s]: 136 B
constexpr int AS = kC + 4;          // fp32 row stride of A and of T during the inversion
constexpr int kSlowBatch = 16;      // slow channels staged per pass
constexpr float kFastFloor = 0x1p-96f;
constexpr float kLogFloor = -1000.0f;   // log2 of a zero decay: exp2 of it is exactly 0 in fp32

struct KdaLds {
  __bf16 qt[kC * QS];               // Q~ = gamma * q          [t][c]
  __bf16 kt[kC * QS];               // K~ = gamma * k          [t][c]
  union {
    __bf16 kr[kC * RS];             // K_R = k / gamma (0 for slow channels)   [t][c]
    float tf[kC * AS];              // T = (I + A)^-1 in fp32 while it is built
    __bf16 ob[kC * RS];             // the block's output rows, staged for 16-byte stores
  };
  __bf16 kbt[kD * CS];              // Kbar^T                  [c][t]
  __bf16 v[kC * VS];                // V                       [t][j]
  union {
    float a[kC * AS];               // A (beta-scaled, strictly lower)
    struct {                        // slow channels of one batch, log2-space
      float g[kSlowBatch][kC];
      float k[kSlowBatch][kC];
      float q[kSlowBatch][kC];
    } slow;
  };
  __bf16 pm[kC * CS];               // P (lower incl. diagonal)
  __bf16 tm[kC * CS];               // T in bf16
  float x[2][16 * 17];              // 16-block products of the inversion
  float beta[kC];
  float gc[kD];                     // gamma_C per channel
  float qtot[8][kD];                // per-octet decay products
  int slow_list[kD];
};

__device__ __forceinline__ bool kda_meta_ok(const KdaDevPlan& p) {
  return p.hdr->magic == kKdaMagic && p.hdr->serial == p.serial;
}

__device__ __forceinline__ float bf_lo(uint32_t x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float bf_hi(uint32_t x) { return __uint_as_float(x & 0xFFFF0000u); }

__device__ __forceinline__ bf16x8 cat(bf16x4 a, bf16x4 b) {
  return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// A operand whose 8 contraction slots of half-wave hf are the columns base + {0..3, 8..11} of
// row `row` (base already includes 4 * hf): the order in which an accumulator holds them.
__device__ __forceinline__ bf16x8 lds_a_perm(const __bf16* rowp, int base) {
  return cat(*reinterpret_cast<const bf16x4*>(rowp + base), *reinterpret_cast<const bf16x4*>(rowp + base + 8));
}

// The same from an fp32 row, rounded to bf16.
__device__ __forceinline__ bf16x8 lds_a_perm_f32(const float* rowp, int base) {
  const float4 lo = *reinterpret_cast<const float4*>(rowp + base);
  const float4 hi = *reinterpret_cast<const float4*>(rowp + base + 8);
  return bf16x8{static_cast<__bf16>(lo.x), static_cast<__bf16>(lo.y), static_cast<__bf16>(lo.z),
                static_cast<__bf16>(lo.w), static_cast<__bf16>(hi.x), static_cast<__bf16>(hi.y),
                static_cast<__bf16>(hi.z), static_cast<__bf16>(hi.w)};
}

// Registers 8kk .. 8kk+7 of an accumulator tile, rounded to bf16: a B operand in permuted order.
__device__ __forceinline__ bf16x8 acc_to_b(const f32x16& acc, int kk) {
  bf16x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = static_cast<__bf16>(acc[8 * kk + e]);
  return r;
}

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Transposing LDS read: within each group of 16 lanes, lane i receives element i%4 of the 8 bytes
// addressed by lanes 4m + i/4, m = 0..3.
__device__ __forceinline__ bf16x4 lds_read_tr(const __bf16* p) {
  const i16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
  return __builtin_bit_cast(bf16x4, r);
}

// Workgroup barrier for LDS traffic only.  __syncthreads() also drains every outstanding global
// load of the wave (its release fence covers all memory), which would stall on the next block's
// prefetch; every exchange between waves here goes through LDS, so draining this wave's LDS
// operations before the barrier is enough.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Raw inputs of one block, as loaded by one thread: channels 4 cq .. 4 cq + 3 of tokens
// 8 oc .. 8 oc + 7 (alpha, k, q), 32 values of one token (v) and one beta.
struct RawBlock {
  float4 a[8];
  uint2 k[8], q[8];
  uint4 v[4];
  float b;
};

// The next block's inputs are loaded in three groups spread over the current block (alpha; k and q;
// v and beta), so that no single burst fills the memory request queue and stalls the issuing wave.
// Rows past the block's last token re-read its last row (always in bounds) and are replaced by
// neutral values (alpha = 1, k = q = v = 0, beta = 0) when they are consumed: no branches here.
struct RawAddr {
  int64_t tok0;
  int L;
};

__device__ __forceinline__ void load_raw_alpha(RawBlock& r, const float* __restrict__ alpha, RawAddr a,
                                               int64_t tok_stride, int64_t head_off, int tid) {
  const int cq = tid & 31, oc = tid >> 5;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int t = min(8 * oc + i, a.L - 1);
    r.a[i] = *reinterpret_cast<const float4*>(alpha + (a.tok0 + t) * tok_stride + head_off + 4 * cq);
  }
}

__device__ __forceinline__ void load_raw_kq(RawBlock& r, const __bf16* __restrict__ k, const __bf16* __restrict__ q,
                                            RawAddr a, int64_t tok_stride, int64_t head_off, int tid) {
  const int cq = tid & 31, oc = tid >> 5;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int t = min(8 * oc + i, a.L - 1);
    const int64_t base = (a.tok0 + t) * tok_stride + head_off + 4 * cq;
    r.k[i] = *reinterpret_cast<const uint2*>(k + base);
    r.q[i] = *reinterpret_cast<const uint2*>(q + base);
  }
}

__device__ __forceinline__ void load_raw_vb(RawBlock& r, const __bf16* __restrict__ v, const float* __restrict__ beta,
                                            RawAddr a, int64_t tok_stride, int64_t head_off, int head, int H, int tid) {
  const int tv = min(tid >> 2, a.L - 1), part = tid & 3;
  // lane `part` of a row takes its 16-byte chunks part + 4u: the four lanes of a row read (and later
  // write to LDS) 64 contiguous bytes per u
  const uint4* src = reinterpret_cast<const uint4*>(v + (a.tok0 + tv) * tok_stride + head_off + 8 * part);
#pragma unroll
  for (int u = 0; u < 4; ++u) r.v[u] = src[4 * u];
  r.b = beta[(a.tok0 + min(tid, a.L - 1)) * H + head];
}

__global__ __launch_bounds__(256, 1) void kda_prefill_kernel(KdaDevPlan p, const __bf16* __restrict__ q,
                                                             const __bf16* __restrict__ k,
                                                             const __bf16* __restrict__ v,
                                                             const float* __restrict__ alpha,
                                                             const float* __restrict__ beta,
                                                             float* __restrict__ state_pool,
                                                             __bf16* __restrict__ out) {
  __shared__ __attribute__((aligned(16))) KdaLds ls;
  if (!kda_meta_ok(p)) return;
  const int H = p.num_heads;
  const int item_idx = blockIdx.x / H, head = blockIdx.x - item_idx * H;
  if (item_idx >= p.num_items) return;
  const KdaItem it = p.items[item_idx];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, col = lane & 31, hf = lane >> 5;
  const int64_t tok_stride = int64_t(H) * kD;           // elements between tokens of one head
  const int64_t head_off = int64_t(head) * kD;
  const int j0 = 32 * wave;                             // this wave's state columns
  const int cq = tid & 31, oc = tid >> 5;               // phase 0: channels 4 cq + e, tokens 8 oc + i

  // ---- state S0 (fp32) -------------------------------------------------------------------------
  // tile ib, register 4b + r: row i = 32 ib + 8 b + 4 hf + r, column j0 + col
  f32x16 S[4];
#pragma unroll
  for (int ib = 0; ib < 4; ++ib) S[ib] = f32x16{};
  if (it.state_in >= 0) {
    const float* src = state_pool + (int64_t(it.state_in) * H + head) * kD * kD + j0 + col;
#pragma unroll
    for (int ib = 0; ib < 4; ++ib)
#pragma unroll
      for (int reg = 0; reg < 16; ++reg)
        S[ib][reg] = src[int64_t(32 * ib + 8 * (reg >> 2) + 4 * hf + (reg & 3)) * kD];
  }

  RawBlock raw;
  {
    const RawAddr first{int64_t(it.cu), min(kC, it.len)};
    load_raw_alpha(raw, alpha, first, tok_stride, head_off, tid);
    load_raw_kq(raw, k, q, first, tok_stride, head_off, tid);
    load_raw_vb(raw, v, beta, first, tok_stride, head_off, head, H, tid);
  }

  for (int blk = 0; blk < it.len; blk += kC) {
    const int L = min(kC, it.len - blk);
    const int64_t tok0 = int64_t(it.cu) + blk;

    // ================= phase 0: decays, scaled operands, V, beta ================================
    float g[8][4];                 // running decay product within the octet, inclusive
    float sfx[8][4];               // decay product of the later tokens of the octet, exclusive
    {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (8 * oc + i >= L) {     // rows past the end: neutral
          raw.a[i] = make_float4(1.0f, 1.0f, 1.0f, 1.0f);
          raw.k[i] = make_uint2(0, 0);
          raw.q[i] = make_uint2(0, 0);
        }
      float run[4] = {1.0f, 1.0f, 1.0f, 1.0f}, back[4] = {1.0f, 1.0f, 1.0f, 1.0f};
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float ai[4] = {raw.a[i].x, raw.a[i].y, raw.a[i].z, raw.a[i].w};
        const float aj[4] = {raw.a[7 - i].x, raw.a[7 - i].y, raw.a[7 - i].z, raw.a[7 - i].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          run[e] *= ai[e];
          g[i][e] = run[e];
          sfx[7 - i][e] = back[e];
          back[e] *= aj[e];
        }
      }
      *reinterpret_cast<float4*>(&ls.qtot[oc][4 * cq]) = make_float4(run[0], run[1], run[2], run[3]);
      const int tv = tid >> 2, part = tid & 3;
      const bool vok = tv < L;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        *reinterpret_cast<uint4*>(&ls.v[tv * VS + 8 * part + 32 * u]) = vok ? raw.v[u] : make_uint4(0, 0, 0, 0);
      if (tid < kC) ls.beta[tid] = tid < L ? raw.b : 0.0f;
    }
    lds_barrier();

    float tot[4], pre[4], post[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      tot[e] = 1.0f;
      pre[e] = 1.0f;
      post[e] = 1.0f;
    }
#pragma unroll
    for (int o = 0; o < 8; ++o) {
      const float4 x = *reinterpret_cast<const float4*>(&ls.qtot[o][4 * cq]);
      const float xs[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (o < oc) pre[e] *= xs[e];
        if (o > oc) post[e] *= xs[e];
        tot[e] *= xs[e];
      }
    }
    // gamma_t = pre * g, gamma_C / gamma_t = sfx * post (a product of the later decays, no division),
    // and k / gamma_t = (k gamma_C / gamma_t) / gamma_C: one reciprocal per channel
    bool slow[4];
    float inv_tot[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      slow[e] = !(tot[e] >= kFastFloor);
      inv_tot[e] = slow[e] ? 0.0f : __frcp_rn(tot[e]);
    }
    {
      __bf16 kb[4][8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int t = 8 * oc + i;
        const float kf[4] = {bf_lo(raw.k[i].x), bf_hi(raw.k[i].x), bf_lo(raw.k[i].y), bf_hi(raw.k[i].y)};
        const float qf[4] = {bf_lo(raw.q[i].x), bf_hi(raw.q[i].x), bf_lo(raw.q[i].y), bf_hi(raw.q[i].y)};
        bf16x4 vq, vk, vr;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float gm = pre[e] * g[i][e];
          vq[e] = static_cast<__bf16>(qf[e] * gm);
          vk[e] = static_cast<__bf16>(kf[e] * gm);
          const float kbar = slow[e] ? 0.0f : kf[e] * (sfx[i][e] * post[e]);
          vr[e] = static_cast<__bf16>(kbar * inv_tot[e]);
          kb[e][i] = static_cast<__bf16>(kbar);
        }
        *reinterpret_cast<bf16x4*>(&ls.qt[t * QS + 4 * cq]) = vq;
        *reinterpret_cast<bf16x4*>(&ls.kt[t * QS + 4 * cq]) = vk;
        *reinterpret_cast<bf16x4*>(&ls.kr[t * RS + 4 * cq]) = vr;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        __bf16* kp = &ls.kbt[(4 * cq + e) * CS + 8 * oc];
        *reinterpret_cast<bf16x4*>(kp) = bf16x4{kb[e][0], kb[e][1], kb[e][2], kb[e][3]};
        *reinterpret_cast<bf16x4*>(kp + 4) = bf16x4{kb[e][4], kb[e][5], kb[e][6], kb[e][7]};
      }
      if (oc == 0) *reinterpret_cast<float4*>(&ls.gc[4 * cq]) = make_float4(tot[0], tot[1], tot[2], tot[3]);
    }
    // compact list of the slow channels, in channel order (lanes 0-31 of every wave see all channels)
    int nslow = 0;
    {
      const uint64_t lo32 = (lane < 32) ? ((lane == 0) ? 0ull : (~0ull >> (64 - lane))) : 0ull;
      int below = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint64_t b = __ballot(slow[e] && lane < 32);
        below += __popcll(b & lo32);
        nslow += __popcll(b);
      }
      if (wave == 0 && lane < 32) {
        int idx = below;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (slow[e]) ls.slow_list[idx++] = 4 * cq + e;
      }
    }
    lds_barrier();

    // ================= phase 1: A and P (waves 0-2: tiles (0,0), (1,0), (1,1)) ====================
    // the next block's inputs arrive while this block is computed (first group here)
    const bool more = blk + kC < it.len;
    const RawAddr next{tok0 + kC, min(kC, it.len - blk - kC)};
    if (more) load_raw_alpha(raw, alpha, next, tok_stride, head_off, tid);
    const int tb1 = wave == 0 ? 0 : 1, sb1 = wave == 2 ? 1 : 0;
    f32x16 accA = {}, accP = {};
    if (wave < 3) {
      // the operands of step kc + 1 are read while step kc's two products run
      const __bf16* kp = &ls.kt[(32 * tb1 + col) * QS + 8 * hf];
      const __bf16* qp = &ls.qt[(32 * tb1 + col) * QS + 8 * hf];
      const __bf16* rp = &ls.kr[(32 * sb1 + col) * RS + 8 * hf];
      auto ld4 = [](const __bf16* p) { return cat(*reinterpret_cast<const bf16x4*>(p), *reinterpret_cast<const bf16x4*>(p + 4)); };
      bf16x8 ak = ld4(kp), aq = ld4(qp), b = *reinterpret_cast<const bf16x8*>(rp);
#pragma unroll
      for (int kc = 0; kc < kD / 16; ++kc) {
        bf16x8 nk = ak, nq = aq, nb = b;
        if (kc + 1 < kD / 16) {
          nk = ld4(kp + 16 * (kc + 1));
          nq = ld4(qp + 16 * (kc + 1));
          nb = *reinterpret_cast<const bf16x8*>(rp + 16 * (kc + 1));
        }
        accA = mfma(ak, b, accA);
        accP = mfma(aq, b, accP);
        ak = nk;
        aq = nq;
        b = nb;
      }
      // keep the scheduler from sinking the reads back next to their products
      __builtin_amdgcn_sched_group_barrier(0x100, 5, 0);
#pragma unroll
      for (int i = 0; i < kD / 16 - 1; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x100, 5, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    }
    // slow channels: exact pairwise terms in log2 space, 16 channels per batch, re-read from memory
    for (int base = 0; base < nslow; base += kSlowBatch) {
      lds_barrier();
      const int cl = tid >> 4, tg = tid & 15;
      const bool have = base + cl < nslow;
      const int ch = have ? ls.slow_list[base + cl] : 0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int t = 4 * tg + u;
        float lg = 0.0f, kv = 0.0f, qv = 0.0f;
        if (have && t < L) {
          const int64_t idx = (tok0 + t) * tok_stride + head_off + ch;
          const float a1 = alpha[idx];
          lg = a1 > 0.0f ? fmaxf(__log2f(a1), kLogFloor) : kLogFloor;
          kv = static_cast<float>(k[idx]);
          qv = static_cast<float>(q[idx]);
        }
        ls.slow.g[cl][t] = lg;
        ls.slow.k[cl][t] = kv;
        ls.slow.q[cl][t] = qv;
      }
      lds_barrier();
      if (tid < kSlowBatch) {
        float run = 0.0f;
        for (int t = 0; t < kC; ++t) {
          run += ls.slow.g[tid][t];
          ls.slow.g[tid][t] = run;
        }
      }
      lds_barrier();
      if (have) {
        const float gC = ls.slow.g[cl][kC - 1];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int t = 4 * tg + u;
          ls.kbt[ch * CS + t] = static_cast<__bf16>(ls.slow.k[cl][t] * exp2f(gC - ls.slow.g[cl][t]));
        }
      }
      if (wave < 3) {
        const int nb = min(kSlowBatch, nslow - base);
        const int s = 32 * sb1 + col;
        for (int c = 0; c < nb; ++c) {
          const float gs = ls.slow.g[c][s], ks = ls.slow.k[c][s];
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) {
            const int t = 32 * tb1 + 8 * (reg >> 2) + 4 * hf + (reg & 3);
            const float e = exp2f(fminf(ls.slow.g[c][t] - gs, 0.0f)) * ks;
            accA[reg] += ls.slow.k[c][t] * e;
            accP[reg] += ls.slow.q[c][t] * e;
          }
        }
      }
    }
    if (nslow > 0) lds_barrier();   // the batch scratch shares storage with A
    if (wave < 3) {
      const int s = 32 * sb1 + col;
      float4 btv[4];
#pragma unroll
      for (int b = 0; b < 4; ++b) btv[b] = *reinterpret_cast<const float4*>(&ls.beta[32 * tb1 + 8 * b + 4 * hf]);
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int t0 = 32 * tb1 + 8 * b + 4 * hf;
        const float bs[4] = {btv[b].x, btv[b].y, btv[b].z, btv[b].w};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = t0 + r;
          ls.a[t * AS + s] = s < t ? accA[4 * b + r] * bs[r] : 0.0f;
          ls.pm[t * CS + s] = static_cast<__bf16>(s <= t ? accP[4 * b + r] : 0.0f);
        }
      }
    }
    lds_barrier();

    // ================= phase 2: T = (I + A)^-1 ==================================================
    if (more) load_raw_kq(raw, k, q, next, tok_stride, head_off, tid);
    {
      // diagonal 16 x 16 blocks by forward substitution: wave -> block, lane -> column
      const int a0 = 16 * wave, jc = lane & 15;
      float xs[16];
      // row t + 1 of the block is read while row t is solved
      float4 rc[4] = {}, rn[4] = {};
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        if (t + 1 < 16) {
#pragma unroll
          for (int k = 0; k < 4; ++k)
            if (4 * k < t + 1) rn[k] = *reinterpret_cast<const float4*>(&ls.a[(a0 + t + 1) * AS + a0 + 4 * k]);
        }
        float acc = (t == jc) ? 1.0f : 0.0f;
#pragma unroll
        for (int u = 0; u < t; ++u) {
          const float4 r = rc[u >> 2];
          const float c = (u & 3) == 0 ? r.x : (u & 3) == 1 ? r.y : (u & 3) == 2 ? r.z : r.w;
          acc -= c * xs[u];
        }
        xs[t] = acc;
#pragma unroll
        for (int k = 0; k < 4; ++k) rc[k] = rn[k];
      }
      if (lane < 16) {
#pragma unroll
        for (int t = 0; t < 16; ++t) ls.tf[(a0 + t) * AS + a0 + jc] = xs[t];
        // the block right of an even diagonal block lies above the diagonal of its 32 x 32 block
        if ((wave & 1) == 0) {
#pragma unroll
          for (int t = 0; t < 16; ++t) ls.tf[(a0 + t) * AS + a0 + 16 + jc] = 0.0f;
        }
      }
    }
    lds_barrier();
    {
      // 16 -> 32: T_ab = -D_a A_ab D_b for (a, b) = (1, 0) and (3, 2); two elements per thread
      const int which = tid >> 7, e = tid & 127, tr = e >> 3, jc = 2 * (e & 7);
      const int ba = 2 * which + 1, bb = 2 * which;
      float x0 = 0.0f, x1 = 0.0f;
      {
        // all sixteen (A, D) pairs are read before the sums start
        float av[16];
        float2 d[16];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const float4 a4 = *reinterpret_cast<const float4*>(&ls.a[(16 * ba + tr) * AS + 16 * bb + 4 * k]);
          av[4 * k] = a4.x;
          av[4 * k + 1] = a4.y;
          av[4 * k + 2] = a4.z;
          av[4 * k + 3] = a4.w;
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) d[u] = *reinterpret_cast<const float2*>(&ls.tf[(16 * bb + u) * AS + 16 * bb + jc]);
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          x0 += av[u] * d[u].x;
          x1 += av[u] * d[u].y;
        }
      }
      ls.x[which][tr * 17 + jc] = x0;
      ls.x[which][tr * 17 + jc + 1] = x1;
      lds_barrier();
      float y0 = 0.0f, y1 = 0.0f;
      {
        float dv[16], xa[16], xb[16];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const float4 d4 = *reinterpret_cast<const float4*>(&ls.tf[(16 * ba + tr) * AS + 16 * ba + 4 * k]);
          dv[4 * k] = d4.x;
          dv[4 * k + 1] = d4.y;
          dv[4 * k + 2] = d4.z;
          dv[4 * k + 3] = d4.w;
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          xa[u] = ls.x[which][u * 17 + jc];
          xb[u] = ls.x[which][u * 17 + jc + 1];
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          y0 -= dv[u] * xa[u];
          y1 -= dv[u] * xb[u];
        }
      }
      ls.tf[(16 * ba + tr) * AS + 16 * bb + jc] = y0;
      ls.tf[(16 * ba + tr) * AS + 16 * bb + jc + 1] = y1;
    }
    lds_barrier();
    if (wave == 0) {
      // 32 -> 64 on the matrix cores: T21 = -T2 (A21 T1)
      f32x16 xacc = {};
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const float* arow = &ls.a[(32 + col) * AS + 16 * kk + 8 * hf];
        const float4 lo = *reinterpret_cast<const float4*>(arow), hi = *reinterpret_cast<const float4*>(arow + 4);
        const bf16x8 aop{static_cast<__bf16>(lo.x), static_cast<__bf16>(lo.y), static_cast<__bf16>(lo.z),
                         static_cast<__bf16>(lo.w), static_cast<__bf16>(hi.x), static_cast<__bf16>(hi.y),
                         static_cast<__bf16>(hi.z), static_cast<__bf16>(hi.w)};
        bf16x8 bop;
#pragma unroll
        for (int e = 0; e < 8; ++e) bop[e] = static_cast<__bf16>(ls.tf[(16 * kk + 8 * hf + e) * AS + col]);
        xacc = mfma(aop, bop, xacc);
      }
      f32x16 yacc = {};
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
        yacc = mfma(lds_a_perm_f32(&ls.tf[(32 + col) * AS + 32], 16 * kk + 4 * hf), acc_to_b(xacc, kk), yacc);
#pragma unroll
      for (int reg = 0; reg < 16; ++reg) {
        const int m = 8 * (reg >> 2) + 4 * hf + (reg & 3);
        ls.tm[(32 + m) * CS + col] = static_cast<__bf16>(-yacc[reg]);
      }
    } else {
      // diagonal 32-blocks to bf16 (zero above the diagonal 16-blocks): 2 x 32 rows x 4 segments of 8
      for (int sgi = tid - 64; sgi < 256; sgi += 192) {
        const int blk32 = sgi >> 7, row = (sgi >> 2) & 31, seg = sgi & 3;
        const int t = 32 * blk32 + row, s0 = 32 * blk32 + 8 * seg;
        bf16x8 w;
#pragma unroll
        for (int e = 0; e < 8; ++e) w[e] = static_cast<__bf16>(((s0 + e) >> 4) <= (t >> 4) ? ls.tf[t * AS + s0 + e] : 0.0f);
        *reinterpret_cast<bf16x4*>(&ls.tm[t * CS + s0]) = bf16x4{w[0], w[1], w[2], w[3]};
        *reinterpret_cast<bf16x4*>(&ls.tm[t * CS + s0 + 4]) = bf16x4{w[4], w[5], w[6], w[7]};
      }
    }
    lds_barrier();

    // ================= phase 3: the state chain (wave -> 32 state columns) =======================
    if (more) load_raw_vb(raw, v, beta, next, tok_stride, head_off, head, H, tid);
    {
      bf16x8 sB[4][2];
#pragma unroll
      for (int ib = 0; ib < 4; ++ib) {
        sB[ib][0] = acc_to_b(S[ib], 0);
        sB[ib][1] = acc_to_b(S[ib], 1);
      }
      f32x16 accE[2] = {}, accO[2] = {};
      {
        // software-pipelined: the A operands of step n + 1 are read while step n's MFMAs run
        bf16x8 ak = lds_a_perm(&ls.kt[col * QS], 4 * hf);
        bf16x8 aq = lds_a_perm(&ls.qt[col * QS], 4 * hf);
#pragma unroll
        for (int n = 0; n < 16; ++n) {
          const int ib = n >> 2, kk = (n >> 1) & 1, tb = n & 1;
          bf16x8 nk = ak, nq = aq;
          if (n + 1 < 16) {
            const int m = n + 1;
            const int cb = 32 * (m >> 2) + 16 * ((m >> 1) & 1) + 4 * hf;
            nk = lds_a_perm(&ls.kt[(32 * (m & 1) + col) * QS], cb);
            nq = lds_a_perm(&ls.qt[(32 * (m & 1) + col) * QS], cb);
          }
          accE[tb] = mfma(ak, sB[ib][kk], accE[tb]);
          accO[tb] = mfma(aq, sB[ib][kk], accO[tb]);
          ak = nk;
          aq = nq;
        }
      }
      // R = beta (V - E), in place in accE.  V[t0 + r][j] for r = 0..3 comes from the transposing
      // read: lane 4m + g of each 16-lane group addresses row t0 + m at column 4g of its group.
      const int j = j0 + col;
      const int grp = lane >> 4, li = lane & 15;
      const int jg = j0 + 16 * (grp & 1) + 4 * (li & 3);
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        // the four V fragments and betas of a block row are read before any is used
        bf16x4 vv[4];
        float4 bt[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int t0 = 32 * tb + 8 * b + 4 * hf;
          vv[b] = lds_read_tr(&ls.v[(t0 + (li >> 2)) * VS + jg]);
          bt[b] = *reinterpret_cast<const float4*>(&ls.beta[t0]);
        }
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const float bs[4] = {bt[b].x, bt[b].y, bt[b].z, bt[b].w};
#pragma unroll
          for (int r = 0; r < 4; ++r)
            accE[tb][4 * b + r] = bs[r] * (static_cast<float>(vv[b][r]) - accE[tb][4 * b + r]);
        }
      }
      bf16x8 rB[2][2];
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        rB[tb][0] = acc_to_b(accE[tb], 0);
        rB[tb][1] = acc_to_b(accE[tb], 1);
      }
      // U = T R (T lower-triangular: block row tb uses block columns sb <= tb).  The six products
      // run in the order (tb, sb, kk) = (0,0,0) (0,0,1) (1,0,0) (1,0,1) (1,1,0) (1,1,1); each A
      // operand is read while the previous product runs.  O += P U below uses the same order.
      f32x16 accU[2] = {};
      {
        bf16x8 a = lds_a_perm(&ls.tm[col * CS], 4 * hf);
#pragma unroll
        for (int n = 0; n < 6; ++n) {
          const int tb = n < 2 ? 0 : 1, sb = n < 4 ? 0 : 1, kk = n & 1;
          bf16x8 na = a;
          if (n + 1 < 6) {
            const int m = n + 1;
            na = lds_a_perm(&ls.tm[(32 * (m < 2 ? 0 : 1) + col) * CS], 32 * (m < 4 ? 0 : 1) + 16 * (m & 1) + 4 * hf);
          }
          accU[tb] = mfma(a, rB[sb][kk], accU[tb]);
          a = na;
        }
      }
      bf16x8 uB[2][2];
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        uB[tb][0] = acc_to_b(accU[tb], 0);
        uB[tb][1] = acc_to_b(accU[tb], 1);
      }
      // O += P U, then store the valid rows
      {
        bf16x8 a = lds_a_perm(&ls.pm[col * CS], 4 * hf);
#pragma unroll
        for (int n = 0; n < 6; ++n) {
          const int tb = n < 2 ? 0 : 1, sb = n < 4 ? 0 : 1, kk = n & 1;
          bf16x8 na = a;
          if (n + 1 < 6) {
            const int m = n + 1;
            na = lds_a_perm(&ls.pm[(32 * (m < 2 ? 0 : 1) + col) * CS], 32 * (m < 4 ? 0 : 1) + 16 * (m & 1) + 4 * hf);
          }
          accO[tb] = mfma(a, uB[sb][kk], accO[tb]);
          a = na;
        }
      }
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
#pragma unroll
        for (int reg = 0; reg < 16; ++reg) {
          const int t = 32 * tb + 8 * (reg >> 2) + 4 * hf + (reg & 3);
          ls.ob[t * RS + j] = static_cast<__bf16>(accO[tb][reg]);
        }
      }
      // S = Diag(gamma_C) S + Kbar^T U: 16 products in the order (ib, sb, kk), each A operand read
      // while the previous product runs
      {
        bf16x8 a = lds_a_perm(&ls.kbt[col * CS], 4 * hf);
        // the decays of block row ib + 1 are read while block row ib is updated
        float4 gcur[4], gnxt[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) gcur[b] = *reinterpret_cast<const float4*>(&ls.gc[8 * b + 4 * hf]);
#pragma unroll
        for (int n = 0; n < 16; ++n) {
          const int ib = n >> 2, sb = (n >> 1) & 1, kk = n & 1;
          if ((n & 3) == 0) {
            if (ib + 1 < 4) {
#pragma unroll
              for (int b = 0; b < 4; ++b)
                gnxt[b] = *reinterpret_cast<const float4*>(&ls.gc[32 * (ib + 1) + 8 * b + 4 * hf]);
            }
#pragma unroll
            for (int b = 0; b < 4; ++b) {
              S[ib][4 * b + 0] *= gcur[b].x;
              S[ib][4 * b + 1] *= gcur[b].y;
              S[ib][4 * b + 2] *= gcur[b].z;
              S[ib][4 * b + 3] *= gcur[b].w;
              gcur[b] = gnxt[b];
            }
          }
          bf16x8 na = a;
          if (n + 1 < 16) {
            const int m = n + 1;
            na = lds_a_perm(&ls.kbt[(32 * (m >> 2) + col) * CS], 32 * ((m >> 1) & 1) + 16 * (m & 1) + 4 * hf);
          }
          S[ib] = mfma(a, uB[sb][kk], S[ib]);
          a = na;
        }
      }
    }
    lds_barrier();
    // the block's output rows leave from LDS as 16-byte stores (the next block writes this storage
    // only after its first barrier)
    {
      const int t = tid >> 2, part = tid & 3;
      if (t < L) {
        uint4* dst = reinterpret_cast<uint4*>(out + (tok0 + t) * tok_stride + head_off + 32 * part);
#pragma unroll
        for (int u = 0; u < 4; ++u) dst[u] = *reinterpret_cast<const uint4*>(&ls.ob[t * RS + 32 * part + 8 * u]);
      }
    }
  }

  // ---- snapshot at the chunk boundary ---------------------------------------------------------
  {
    float* dst = state_pool + (int64_t(it.state_out) * H + head) * kD * kD + j0 + col;
#pragma unroll
    for (int ib = 0; ib < 4; ++ib)
#pragma unroll
      for (int reg = 0; reg < 16; ++reg) {
        const int i = 32 * ib + 8 * (reg >> 2) + 4 * hf + (reg & 3);
        dst[int64_t(i) * kD] = S[ib][reg];
      }
  }
}


}  // namespace

hipError_t launch_kda_prefill(const KdaDevPlan& p, const void* q, const void* k, const void* v, const float* alpha,
                              const float* beta, float* state_pool, void* out, hipStream_t stream) {
  if (p.num_items == 0) return hipSuccess;
  const dim3 grid(p.num_items * p.num_heads), block(256);
  hipLaunchKernelGGL(kda_prefill_kernel, grid, block, 0, stream, p, static_cast<const __bf16*>(q),
                     static_cast<const __bf16*>(k), static_cast<const __bf16*>(v), alpha, beta, state_pool,
                     static_cast<__bf16*>(out));
  return hipGetLastError();
}

}  // namespace wavepp
