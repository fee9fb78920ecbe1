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
// when its block decay gamma_C is at least 2^-96, so every factor stays a normal number.  A
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

constexpr int kC = kKdaBlock;       // tokens per block
constexpr int kD = kKdaDim;         // d_k = d_v
constexpr int RS = kD + 8;          // bf16 row stride of token-major [t][channel] arrays
constexpr int CS = kC + 8;          // bf16 row stride of [channel][t] arrays and of P, T [t][s]
constexpr int AS = kC + 4;          // fp32 row stride of A and of T during the inversion
constexpr int kSlowBatch = 16;      // slow channels staged per pass
constexpr float kFastFloor = 0x1p-96f;
constexpr float kLogFloor = -1000.0f;   // log2 of a zero decay: exp2 of it is exactly 0 in fp32

struct KdaLds {
  __bf16 qt[kC * RS];               // Q~ = gamma * q          [t][c]
  __bf16 kt[kC * RS];               // K~ = gamma * k          [t][c]
  union {
    __bf16 kr[kC * RS];             // K_R = k / gamma (0 for slow channels)   [t][c]
    float tf[kC * AS];              // T = (I + A)^-1 in fp32 while it is built
  };
  __bf16 kbt[kD * CS];              // Kbar^T                  [c][t]
  __bf16 vt[kD * CS];               // V^T                     [j][t]
  float a[kC * AS];                 // A (beta-scaled, strictly lower)
  __bf16 pm[kC * CS];               // P (lower incl. diagonal)
  __bf16 tm[kC * CS];               // T in bf16
  float x[3][16 * 17];              // block products of the inversion
  float beta[kC];
  float gc[kD];                     // gamma_C per channel
  float qtot[4][kD];                // per-quarter decay products
  float ltot[4][kD];                // per-quarter log2-decay sums (slow channels)
  float slow_g[kSlowBatch][kC];
  float slow_k[kSlowBatch][kC];
  float slow_q[kSlowBatch][kC];
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

  // ---- state S0 (fp32) -------------------------------------------------------------------------
  // tile ib, register 4b + r: row i = 32 ib + 8 b + 4 hf + r, column j0 + col
  f32x16 S[4];
  {
    const float* src = state_pool + (int64_t(it.state_in) * H + head) * kD * kD + j0 + col;
#pragma unroll
    for (int ib = 0; ib < 4; ++ib)
#pragma unroll
      for (int reg = 0; reg < 16; ++reg) {
        const int i = 32 * ib + 8 * (reg >> 2) + 4 * hf + (reg & 3);
        S[ib][reg] = it.state_in >= 0 ? src[int64_t(i) * kD] : 0.0f;
      }
  }

  const int ch0 = 2 * lane;        // phase-0 channels of this thread: ch0, ch0 + 1
  const int qq = wave;             // phase-0 token quarter: [16 qq, 16 qq + 16)

  for (int blk = 0; blk < it.len; blk += kC) {
    const int L = min(kC, it.len - blk);
    const int64_t tok0 = int64_t(it.cu) + blk;

    // ================= phase 0: decays, scaled operands, V^T, beta ==============================
    float g0[16], g1[16];          // running decay product within the quarter
    uint32_t kraw[16], qraw[16];   // bf16 pairs (ch0, ch0 + 1)
    float run0 = 1.0f, run1 = 1.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int t = 16 * qq + i;
      float2 a2 = make_float2(1.0f, 1.0f);
      uint32_t kr2 = 0, qr2 = 0;
      if (t < L) {
        const int64_t base = (tok0 + t) * tok_stride + head_off + ch0;
        a2 = *reinterpret_cast<const float2*>(alpha + base);
        kr2 = *reinterpret_cast<const uint32_t*>(k + base);
        qr2 = *reinterpret_cast<const uint32_t*>(q + base);
      }
      run0 *= a2.x;
      run1 *= a2.y;
      g0[i] = run0;
      g1[i] = run1;
      kraw[i] = kr2;
      qraw[i] = qr2;
    }
    ls.qtot[qq][ch0] = run0;
    ls.qtot[qq][ch0 + 1] = run1;
    if (tid < kC) ls.beta[tid] = tid < L ? beta[(tok0 + tid) * H + head] : 0.0f;
    {
      // V^T: thread -> (token, 32-column part)
      const int t = tid >> 2, part = tid & 3;
      uint4 raw[4] = {};
      if (t < L) {
        const uint4* src = reinterpret_cast<const uint4*>(v + (tok0 + t) * tok_stride + head_off + 32 * part);
#pragma unroll
        for (int u = 0; u < 4; ++u) raw[u] = src[u];
      }
      const __bf16* e = reinterpret_cast<const __bf16*>(raw);
#pragma unroll
      for (int jj = 0; jj < 32; ++jj) ls.vt[(32 * part + jj) * CS + t] = e[jj];
    }
    __syncthreads();

    float pre0 = 1.0f, pre1 = 1.0f, tot0 = 1.0f, tot1 = 1.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float x0 = ls.qtot[w][ch0], x1 = ls.qtot[w][ch0 + 1];
      if (w < qq) {
        pre0 *= x0;
        pre1 *= x1;
      }
      tot0 *= x0;
      tot1 *= x1;
    }
    const bool slow0 = !(tot0 >= kFastFloor), slow1 = !(tot1 >= kFastFloor);
    const int any_slow = __syncthreads_or(int(slow0 || slow1));

    // log2-space decays of slow channels
    float lg0[16], lg1[16], G0pre = 0.0f, G1pre = 0.0f, G0C = 0.0f, G1C = 0.0f;
    int nslow = 0, idx0 = 0, idx1 = 0;
    if (any_slow) {
      float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int t = 16 * qq + i;
        float l0 = 0.0f, l1 = 0.0f;
        if (t < L && (slow0 || slow1)) {
          const float2 a2 = *reinterpret_cast<const float2*>(alpha + (tok0 + t) * tok_stride + head_off + ch0);
          l0 = fmaxf(__log2f(a2.x), kLogFloor);
          l1 = fmaxf(__log2f(a2.y), kLogFloor);
          if (!(a2.x > 0.0f)) l0 = kLogFloor;
          if (!(a2.y > 0.0f)) l1 = kLogFloor;
        }
        s0 += l0;
        s1 += l1;
        lg0[i] = s0;
        lg1[i] = s1;
      }
      ls.ltot[qq][ch0] = s0;
      ls.ltot[qq][ch0 + 1] = s1;
      __syncthreads();
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float x0 = ls.ltot[w][ch0], x1 = ls.ltot[w][ch0 + 1];
        if (w < qq) {
          G0pre += x0;
          G1pre += x1;
        }
        G0C += x0;
        G1C += x1;
      }
      // compact index of the slow channels, in channel order (every wave sees all channels)
      const uint64_t b0 = __ballot(slow0), b1 = __ballot(slow1);
      const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
      idx0 = __popcll(b0 & below) + __popcll(b1 & below);
      idx1 = idx0 + (slow0 ? 1 : 0);
      nslow = __popcll(b0) + __popcll(b1);
    }

    // scaled operands
    {
      __bf16 kb0[16], kb1[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int t = 16 * qq + i;
        const float gm0 = pre0 * g0[i], gm1 = pre1 * g1[i];
        const float k0 = bf_lo(kraw[i]), k1 = bf_hi(kraw[i]);
        const float q0 = bf_lo(qraw[i]), q1 = bf_hi(qraw[i]);
        *reinterpret_cast<bf16x2*>(&ls.qt[t * RS + ch0]) = bf16x2{static_cast<__bf16>(q0 * gm0), static_cast<__bf16>(q1 * gm1)};
        *reinterpret_cast<bf16x2*>(&ls.kt[t * RS + ch0]) = bf16x2{static_cast<__bf16>(k0 * gm0), static_cast<__bf16>(k1 * gm1)};
        const float r0 = slow0 ? 0.0f : k0 * __frcp_rn(gm0);
        const float r1 = slow1 ? 0.0f : k1 * __frcp_rn(gm1);
        *reinterpret_cast<bf16x2*>(&ls.kr[t * RS + ch0]) = bf16x2{static_cast<__bf16>(r0), static_cast<__bf16>(r1)};
        const float kb0f = slow0 ? k0 * exp2f(G0C - (G0pre + lg0[i])) : r0 * tot0;
        const float kb1f = slow1 ? k1 * exp2f(G1C - (G1pre + lg1[i])) : r1 * tot1;
        kb0[i] = static_cast<__bf16>(kb0f);
        kb1[i] = static_cast<__bf16>(kb1f);
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        *reinterpret_cast<bf16x8*>(&ls.kbt[ch0 * CS + 16 * qq + 8 * u]) =
            bf16x8{kb0[8 * u], kb0[8 * u + 1], kb0[8 * u + 2], kb0[8 * u + 3], kb0[8 * u + 4], kb0[8 * u + 5], kb0[8 * u + 6], kb0[8 * u + 7]};
        *reinterpret_cast<bf16x8*>(&ls.kbt[(ch0 + 1) * CS + 16 * qq + 8 * u]) =
            bf16x8{kb1[8 * u], kb1[8 * u + 1], kb1[8 * u + 2], kb1[8 * u + 3], kb1[8 * u + 4], kb1[8 * u + 5], kb1[8 * u + 6], kb1[8 * u + 7]};
      }
      if (qq == 0) {
        ls.gc[ch0] = tot0;
        ls.gc[ch0 + 1] = tot1;
      }
    }
    __syncthreads();

    // ================= phase 1: A and P (waves 0-2: tiles (0,0), (1,0), (1,1)) ====================
    const int tb1 = wave == 0 ? 0 : 1, sb1 = wave == 2 ? 1 : 0;
    f32x16 accA = {}, accP = {};
    if (wave < 3) {
#pragma unroll
      for (int kc = 0; kc < kD / 16; ++kc) {
        const bf16x8 ak = *reinterpret_cast<const bf16x8*>(&ls.kt[(32 * tb1 + col) * RS + 16 * kc + 8 * hf]);
        const bf16x8 aq = *reinterpret_cast<const bf16x8*>(&ls.qt[(32 * tb1 + col) * RS + 16 * kc + 8 * hf]);
        const bf16x8 b = *reinterpret_cast<const bf16x8*>(&ls.kr[(32 * sb1 + col) * RS + 16 * kc + 8 * hf]);
        accA = mfma(ak, b, accA);
        accP = mfma(aq, b, accP);
      }
    }
    // exact pairwise terms of slow channels, in batches
    for (int base = 0; base < nslow; base += kSlowBatch) {
      __syncthreads();
      if (slow0 && idx0 >= base && idx0 < base + kSlowBatch) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int t = 16 * qq + i;
          ls.slow_g[idx0 - base][t] = G0pre + lg0[i];
          ls.slow_k[idx0 - base][t] = bf_lo(kraw[i]);
          ls.slow_q[idx0 - base][t] = bf_lo(qraw[i]);
        }
      }
      if (slow1 && idx1 >= base && idx1 < base + kSlowBatch) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int t = 16 * qq + i;
          ls.slow_g[idx1 - base][t] = G1pre + lg1[i];
          ls.slow_k[idx1 - base][t] = bf_hi(kraw[i]);
          ls.slow_q[idx1 - base][t] = bf_hi(qraw[i]);
        }
      }
      __syncthreads();
      if (wave < 3) {
        const int nb = min(kSlowBatch, nslow - base);
        const int s = 32 * sb1 + col;
        for (int c = 0; c < nb; ++c) {
          const float gs = ls.slow_g[c][s], ks = ls.slow_k[c][s];
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) {
            const int t = 32 * tb1 + 8 * (reg >> 2) + 4 * hf + (reg & 3);
            const float e = exp2f(fminf(ls.slow_g[c][t] - gs, 0.0f)) * ks;
            accA[reg] += ls.slow_k[c][t] * e;
            accP[reg] += ls.slow_q[c][t] * e;
          }
        }
      }
    }
    if (wave < 3) {
      const int s = 32 * sb1 + col;
#pragma unroll
      for (int reg = 0; reg < 16; ++reg) {
        const int t = 32 * tb1 + 8 * (reg >> 2) + 4 * hf + (reg & 3);
        ls.a[t * AS + s] = s < t ? accA[reg] * ls.beta[t] : 0.0f;
        ls.pm[t * CS + s] = static_cast<__bf16>(s <= t ? accP[reg] : 0.0f);
      }
    }
    __syncthreads();

    // ================= phase 2: T = (I + A)^-1 ==================================================
    {
      // diagonal 16 x 16 blocks by forward substitution: wave -> block, lane -> column
      const int a0 = 16 * wave, jc = lane & 15;
      float xs[16];
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        float acc = (t == jc) ? 1.0f : 0.0f;
#pragma unroll
        for (int u = 0; u < t; ++u) acc -= ls.a[(a0 + t) * AS + a0 + u] * xs[u];
        xs[t] = acc;
      }
      if (lane < 16) {
#pragma unroll
        for (int t = 0; t < 16; ++t) ls.tf[(a0 + t) * AS + a0 + jc] = xs[t];
      }
    }
    __syncthreads();
    {
      // off-diagonal blocks by distance d: T_ab = -D_a sum_{c=b}^{a-1} A_ac T_cb
      const int tr = tid >> 4, jc = tid & 15;
      for (int d = 1; d < 4; ++d) {
        for (int bi = 0; bi < 4 - d; ++bi) {
          const int ba = bi + d, bb = bi;
          float acc = 0.0f;
          for (int c = bb; c < ba; ++c)
#pragma unroll
            for (int u = 0; u < 16; ++u)
              acc += ls.a[(16 * ba + tr) * AS + 16 * c + u] * ls.tf[(16 * c + u) * AS + 16 * bb + jc];
          ls.x[bi][tr * 17 + jc] = acc;
        }
        __syncthreads();
        for (int bi = 0; bi < 4 - d; ++bi) {
          const int ba = bi + d, bb = bi;
          float acc = 0.0f;
#pragma unroll
          for (int u = 0; u < 16; ++u) acc -= ls.tf[(16 * ba + tr) * AS + 16 * ba + u] * ls.x[bi][u * 17 + jc];
          ls.tf[(16 * ba + tr) * AS + 16 * bb + jc] = acc;
        }
        __syncthreads();
      }
      for (int e = tid; e < kC * kC; e += 256) {
        const int t = e >> 6, s = e & 63;
        ls.tm[t * CS + s] = static_cast<__bf16>((s >> 4) <= (t >> 4) ? ls.tf[t * AS + s] : 0.0f);
      }
    }
    __syncthreads();

    // ================= phase 3: the state chain (wave -> 32 state columns) =======================
    {
      bf16x8 sB[4][2];
#pragma unroll
      for (int ib = 0; ib < 4; ++ib) {
        sB[ib][0] = acc_to_b(S[ib], 0);
        sB[ib][1] = acc_to_b(S[ib], 1);
      }
      f32x16 accE[2] = {}, accO[2] = {};
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        const __bf16* ktr = &ls.kt[(32 * tb + col) * RS];
        const __bf16* qtr = &ls.qt[(32 * tb + col) * RS];
#pragma unroll
        for (int ib = 0; ib < 4; ++ib)
#pragma unroll
          for (int kk = 0; kk < 2; ++kk) {
            const int cb = 32 * ib + 16 * kk + 4 * hf;
            accE[tb] = mfma(lds_a_perm(ktr, cb), sB[ib][kk], accE[tb]);
            accO[tb] = mfma(lds_a_perm(qtr, cb), sB[ib][kk], accO[tb]);
          }
      }
      // R = beta (V - E), in place in accE
      const int j = j0 + col;
#pragma unroll
      for (int tb = 0; tb < 2; ++tb)
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int t0 = 32 * tb + 8 * b + 4 * hf;
          const bf16x4 vv = *reinterpret_cast<const bf16x4*>(&ls.vt[j * CS + t0]);
#pragma unroll
          for (int r = 0; r < 4; ++r)
            accE[tb][4 * b + r] = ls.beta[t0 + r] * (static_cast<float>(vv[r]) - accE[tb][4 * b + r]);
        }
      bf16x8 rB[2][2];
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        rB[tb][0] = acc_to_b(accE[tb], 0);
        rB[tb][1] = acc_to_b(accE[tb], 1);
      }
      // U = T R (T lower-triangular: block row tb uses block columns sb <= tb)
      f32x16 accU[2] = {};
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        const __bf16* tr = &ls.tm[(32 * tb + col) * CS];
#pragma unroll
        for (int sb = 0; sb <= tb; ++sb)
#pragma unroll
          for (int kk = 0; kk < 2; ++kk) accU[tb] = mfma(lds_a_perm(tr, 32 * sb + 16 * kk + 4 * hf), rB[sb][kk], accU[tb]);
      }
      bf16x8 uB[2][2];
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        uB[tb][0] = acc_to_b(accU[tb], 0);
        uB[tb][1] = acc_to_b(accU[tb], 1);
      }
      // O += P U, then store the valid rows
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        const __bf16* pr = &ls.pm[(32 * tb + col) * CS];
#pragma unroll
        for (int sb = 0; sb <= tb; ++sb)
#pragma unroll
          for (int kk = 0; kk < 2; ++kk) accO[tb] = mfma(lds_a_perm(pr, 32 * sb + 16 * kk + 4 * hf), uB[sb][kk], accO[tb]);
#pragma unroll
        for (int reg = 0; reg < 16; ++reg) {
          const int t = 32 * tb + 8 * (reg >> 2) + 4 * hf + (reg & 3);
          if (t < L) out[(tok0 + t) * tok_stride + head_off + j] = static_cast<__bf16>(accO[tb][reg]);
        }
      }
      // S = Diag(gamma_C) S + Kbar^T U
#pragma unroll
      for (int ib = 0; ib < 4; ++ib) {
#pragma unroll
        for (int reg = 0; reg < 16; ++reg) S[ib][reg] *= ls.gc[32 * ib + 8 * (reg >> 2) + 4 * hf + (reg & 3)];
        const __bf16* kr = &ls.kbt[(32 * ib + col) * CS];
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
          for (int kk = 0; kk < 2; ++kk) S[ib] = mfma(lds_a_perm(kr, 32 * sb + 16 * kk + 4 * hf), uB[sb][kk], S[ib]);
      }
    }
    __syncthreads();
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
