// Chunkwise WY-form refresh kernel on bf16 MFMA (gfx950), dk = dv = 128.
//
// Same recurrence as the per-column kernel (Sec. 3.1, Eq. 1 on S' = S^T):
//     S~ = Diag(exp(g_t)) S'_{t-1},   S'_t = S~ + beta_t k_t (v_t - S~^T k_t)^T.
// Unrolled over a chunk of C = 32 tokens with G_t = sum_{r<=t} g_r (per channel):
//     A_ts = beta_t sum_c k_tc k_sc exp(G_tc - G_sc)      (s < t)
//     T    = (I + A)^{-1},   T' = T Diag(beta)
//     U    = T' V - (T' K_G) S'          K_G = k * exp(G)          (per-token deltas)
//     S'  <- Diag(exp(G_C)) S' + K_H^T U   K_H = k * exp(G_C - G)
// which is the per-token rule exactly, up to rounding.
//
// Work split: one 256-thread block per (request, head); wave w owns value columns
// [32w, 32w + 32) of S' (128 x 32 fp32 = 16 MFMA accumulator tiles held in VGPRs for
// the whole replay).  The per-chunk quantities that do not depend on S' (cumulative
// decays, A, T', T' K_G, K_H) are built cooperatively in LDS; then each wave runs
// the two state contractions on its columns.
//
// Precision.  Every product runs on v_mfma_f32_16x16x32_bf16 with fp32 accumulation.
// An fp32 operand x is split into x_hi = bf16(x) and x_lo = bf16(x - x_hi); a product
// is formed as a_hi b_hi + a_lo b_hi + a_hi b_lo, which keeps ~16 mantissa bits per
// term (exact bf16 inputs such as v skip the split).  This is what lets an fp32 state
// survive thousands of tokens within 2e-3 while running at bf16 matrix-core rate.
//
// Register-resident chaining.  In the 16x16x32 layout lane (q = lane/16, r = lane%16)
// holds A[m = r][k = 8q + e], B[k = 8q + e][n = r] and D[m = 4q + i][n = r].  The
// contraction index k can be any bijection shared by A and B, so the state tiles
// (D layout: rows 4q + i) are fed straight back as B operands by taking
// k(q, e) = 4q + e (e < 4) and 16 + 4q + (e - 4) (e >= 4) over a pair of 16-row tiles;
// the LDS-side operand is read with the same mapping.  Neither S' nor U ever leaves
// registers.
//
// Decay factors.  exp(G_t - G_s) <= 1 for s <= t, but the factorised form needs
// exp(G_t - G_ref) exp(G_ref - G_s).  Off-diagonal 16-token blocks use the block
// boundary as reference (both factors <= 1); diagonal blocks use the block midpoint,
// whose factors are bounded by exp(8 |g|max).  Per-token log-gates are therefore
// floored at -10 (a decay of 4.5e-5 per token instead of anything smaller), which
// keeps every factor below e^80 in fp32 and changes the state by at most 4.5e-5 of
// its magnitude per floored token.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "refresh_kernels.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int C = 32;       // tokens per chunk
constexpr int D = 128;      // dk = dv
constexpr float kGateFloor = -10.f;

// LDS map (bytes).  G is dead once the A tiles and K_G/K_H are built, and its space
// then holds -T'K_G.
constexpr int OFF_G = 0;            // f32 [C][D] cumulative log-decay
constexpr int OFF_WNH = 0;          // bf16 [C][D] -(T'K_G), hi part
constexpr int OFF_WNL = 8192;       // bf16 [C][D] lo part
constexpr int OFF_KRAW = 16384;     // bf16 [C][D] keys of the chunk
constexpr int OFF_VT = 24576;       // bf16 [D][C] values, transposed
constexpr int OFF_KGH = 32768;      // bf16 [D][C] K_G^T hi
constexpr int OFF_KGL = 40960;      // bf16 [D][C] K_G^T lo
constexpr int OFF_KHH = 49152;      // bf16 [D][C] K_H^T hi
constexpr int OFF_KHL = 57344;      // bf16 [D][C] K_H^T lo
constexpr int OFF_AM = 65536;       // f32 [C][C] A
constexpr int OFF_TM = 69632;       // f32 [C][C] T
constexpr int OFF_Y = 73728;        // f32 [16][16] A10 T00
constexpr int OFF_TPH = 74752;      // bf16 [C][C] T' hi
constexpr int OFF_TPL = 76800;      // bf16 [C][C] T' lo
constexpr int OFF_BETA = 78848;     // f32 [C]
constexpr int OFF_GAM = 78976;      // f32 [D] exp(G_C)
constexpr int LDS_BYTES = 79488;

__device__ inline float bf2f(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

__device__ inline void split(float x, __bf16& hi, __bf16& lo) {
  hi = static_cast<__bf16>(x);
  lo = static_cast<__bf16>(x - static_cast<float>(hi));
}

__device__ inline f32x4 mma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// a b with both operands split: a_lo b_hi + a_hi b_lo + a_hi b_hi (small terms first)
__device__ inline f32x4 mma3(bf16x8 ah, bf16x8 al, bf16x8 bh, bf16x8 bl, f32x4 c) {
  c = mma(al, bh, c);
  c = mma(ah, bl, c);
  return mma(ah, bh, c);
}

__device__ inline bf16x8 cat(bf16x4 a, bf16x4 b) {
  return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

template <bool PER_CHANNEL>
__global__ __launch_bounds__(256, 2) void refresh_wy_kernel(
    int H, int Hqk, int layer, int L, const int32_t* __restrict__ inv_row,
    float* __restrict__ states, int64_t n_pool, const int32_t* __restrict__ slot,
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ v, const float* __restrict__ g,
    const float* __restrict__ beta, int W, int init_zero) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[LDS_BYTES];
  float* sG = reinterpret_cast<float*>(smem + OFF_G);
  __bf16* sWNH = reinterpret_cast<__bf16*>(smem + OFF_WNH);
  __bf16* sWNL = reinterpret_cast<__bf16*>(smem + OFF_WNL);
  uint16_t* sK = reinterpret_cast<uint16_t*>(smem + OFF_KRAW);
  uint16_t* sVT = reinterpret_cast<uint16_t*>(smem + OFF_VT);
  __bf16* sKGH = reinterpret_cast<__bf16*>(smem + OFF_KGH);
  __bf16* sKGL = reinterpret_cast<__bf16*>(smem + OFF_KGL);
  __bf16* sKHH = reinterpret_cast<__bf16*>(smem + OFF_KHH);
  __bf16* sKHL = reinterpret_cast<__bf16*>(smem + OFF_KHL);
  float* sA = reinterpret_cast<float*>(smem + OFF_AM);
  float* sT = reinterpret_cast<float*>(smem + OFF_TM);
  float* sY = reinterpret_cast<float*>(smem + OFF_Y);
  __bf16* sTPH = reinterpret_cast<__bf16*>(smem + OFF_TPH);
  __bf16* sTPL = reinterpret_cast<__bf16*>(smem + OFF_TPL);
  float* sBeta = reinterpret_cast<float*>(smem + OFF_BETA);
  float* sGam = reinterpret_cast<float*>(smem + OFF_GAM);

  const int n = blockIdx.x / H;
  const int h = blockIdx.x - n * H;
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int q = lane >> 4, r = lane & 15;

  const int64_t head_row = (int64_t(layer) * H + h) * D;
  bool mine = false;
  if (tid < D) mine = inv_row[head_row + tid] < 0;
  if (!__syncthreads_or(mine)) return;
  const int64_t sl = slot[n];
  if (sl < 0 || sl >= n_pool) return;
  float* S_head = states + (sl * L * H * D + head_row) * D;

  // S'[c][j] for c = 16 mt + 4q + i, j = 32w + 16 nt + r
  f32x4 S[8][2];
#pragma unroll
  for (int mt = 0; mt < 8; ++mt)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        S[mt][nt][i] = init_zero ? 0.f : S_head[int64_t(16 * mt + 4 * q + i) * D + 32 * w + 16 * nt + r];

  const int hk = h / (H / Hqk);
  const uint16_t* kp = k + (int64_t(n) * Hqk + hk) * W * D;
  const uint16_t* vp = v + (int64_t(n) * H + h) * W * D;
  const float* gp = PER_CHANNEL ? g + (int64_t(n) * H + h) * W * D : g + (int64_t(n) * H + h) * W;
  const float* bp = beta + (int64_t(n) * H + h) * W;

  const int ch = tid & (D - 1);   // channel owned in the decay phases
  const int hf = tid >> 7;        // which 16-token half of the chunk

  for (int t0 = 0; t0 < W; t0 += C) {
    const int nv = min(C, W - t0);  // valid tokens; the rest are zero (identity) tokens

    // ---- load: gates -> cumulative decay, keys, values (transposed), beta ------------
    float Gl[16];
    {
      float run = 0.f;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int t = 16 * hf + i;
        float gv = 0.f;
        if (t < nv) gv = PER_CHANNEL ? gp[int64_t(t0 + t) * D + ch] : gp[t0 + t];
        run += fmaxf(gv, kGateFloor);
        Gl[i] = run;
      }
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int e = tid + 256 * u;
      const int t = e >> 4, c8 = (e & 15) * 8;
      uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
      if (t < nv) {
        kv = *reinterpret_cast<const uint4*>(kp + int64_t(t0 + t) * D + c8);
        vv = *reinterpret_cast<const uint4*>(vp + int64_t(t0 + t) * D + c8);
      }
      *reinterpret_cast<uint4*>(sK + t * D + c8) = kv;
      const uint32_t vw[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        sVT[(c8 + 2 * x) * C + t] = uint16_t(vw[x] & 0xFFFF);
        sVT[(c8 + 2 * x + 1) * C + t] = uint16_t(vw[x] >> 16);
      }
    }
    if (tid < C) sBeta[tid] = tid < nv ? bp[t0 + tid] : 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) sG[(16 * hf + i) * D + ch] = Gl[i];
    __syncthreads();
    if (hf == 1) {
      const float base = sG[15 * D + ch];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        Gl[i] += base;
        sG[(16 + i) * D + ch] = Gl[i];
      }
      sGam[ch] = __expf(Gl[15]);
    }
    __syncthreads();

    // ---- K_G^T = (k exp(G))^T and K_H^T = (k exp(G_C - G))^T, split hi/lo ----------
    {
      const float gC = sG[31 * D + ch];
      bf16x8 gh[2], gl[2], hh[2], hl[2];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float kv = bf2f(sK[(16 * hf + i) * D + ch]);
        __bf16 a, b;
        split(kv * __expf(Gl[i]), a, b);
        gh[i >> 3][i & 7] = a;
        gl[i >> 3][i & 7] = b;
        split(kv * __expf(gC - Gl[i]), a, b);
        hh[i >> 3][i & 7] = a;
        hl[i >> 3][i & 7] = b;
      }
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        const int o = ch * C + 16 * hf + 8 * x;
        *reinterpret_cast<bf16x8*>(sKGH + o) = gh[x];
        *reinterpret_cast<bf16x8*>(sKGL + o) = gl[x];
        *reinterpret_cast<bf16x8*>(sKHH + o) = hh[x];
        *reinterpret_cast<bf16x8*>(sKHL + o) = hl[x];
      }
    }

    // ---- A = Diag(beta) (strictly lower part of R Q^T), three 16x16 tiles -----------
    if (w < 3) {
      const int ti = w == 0 ? 0 : 1, si = w == 2 ? 1 : 0;
      const int rf = w == 0 ? 8 : (w == 1 ? 15 : 24);   // reference token of the tile
      const int tr = 16 * ti + r, sr = 16 * si + r;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int c0 = 32 * kk + 8 * q;
        bf16x8 rh, rl, qh, ql;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float gref = sG[rf * D + c0 + e];
          __bf16 a, b;
          split(bf2f(sK[tr * D + c0 + e]) * __expf(sG[tr * D + c0 + e] - gref), a, b);
          rh[e] = a;
          rl[e] = b;
          split(bf2f(sK[sr * D + c0 + e]) * __expf(gref - sG[sr * D + c0 + e]), a, b);
          qh[e] = a;
          ql[e] = b;
        }
        acc = mma3(rh, rl, qh, ql, acc);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = 16 * ti + 4 * q + i;
        const float val = (ti == si && sr >= t) ? 0.f : sBeta[t] * acc[i];
        sA[t * C + sr] = val;
      }
    }
    __syncthreads();

    // ---- T = (I + A)^{-1}: diagonal 16x16 blocks by forward substitution -----------
    if (w == 0 && lane < 32) {
      const int base = 16 * (lane >> 4), s = lane & 15;
      float x[16];
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        float acc = (t == s) ? 1.f : 0.f;
#pragma unroll
        for (int rr = 0; rr < t; ++rr) acc = fmaf(-sA[(base + t) * C + base + rr], x[rr], acc);
        x[t] = acc;
        sT[(base + t) * C + base + s] = acc;
      }
    }
    __syncthreads();
    {  // Y = A10 T00
      const int t = tid >> 4, s = tid & 15;
      float acc = 0.f;
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) acc = fmaf(sA[(16 + t) * C + rr], sT[rr * C + s], acc);
      sY[t * 16 + s] = acc;
    }
    __syncthreads();
    {  // T10 = -T11 Y
      const int t = tid >> 4, s = tid & 15;
      float acc = 0.f;
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) acc = fmaf(sT[(16 + t) * C + 16 + rr], sY[rr * 16 + s], acc);
      sT[(16 + t) * C + s] = -acc;
    }
    __syncthreads();
    // T' = T Diag(beta), lower triangle only, split hi/lo
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = tid + 256 * u;
      const int t = e >> 5, s = e & 31;
      const float val = s <= t ? sT[e] * sBeta[s] : 0.f;
      __bf16 a, b;
      split(val, a, b);
      sTPH[e] = a;
      sTPL[e] = b;
    }
    __syncthreads();

    // ---- -(T' K_G) computed transposed: rows = channels of this wave's 32 ------------
#pragma unroll
    for (int mtw = 0; mtw < 2; ++mtw) {
      const int cr = 32 * w + 16 * mtw + r;
      const bf16x8 ah = *reinterpret_cast<const bf16x8*>(sKGH + cr * C + 8 * q);
      const bf16x8 al = *reinterpret_cast<const bf16x8*>(sKGL + cr * C + 8 * q);
#pragma unroll
      for (int ntw = 0; ntw < 2; ++ntw) {
        const int tr = 16 * ntw + r;
        const bf16x8 bh = *reinterpret_cast<const bf16x8*>(sTPH + tr * C + 8 * q);
        const bf16x8 bl = *reinterpret_cast<const bf16x8*>(sTPL + tr * C + 8 * q);
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        acc = mma3(ah, al, bh, bl, acc);
        bf16x4 oh, ol;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          __bf16 a, b;
          split(-acc[i], a, b);
          oh[i] = a;
          ol[i] = b;
        }
        const int o = tr * D + 32 * w + 16 * mtw + 4 * q;
        *reinterpret_cast<bf16x4*>(sWNH + o) = oh;
        *reinterpret_cast<bf16x4*>(sWNL + o) = ol;
      }
    }
    __syncthreads();

    // ---- U = T'V - (T'K_G) S' on this wave's columns -----------------------------------
    f32x4 U[2][2];
#pragma unroll
    for (int mu = 0; mu < 2; ++mu) {
      const bf16x8 ah = *reinterpret_cast<const bf16x8*>(sTPH + (16 * mu + r) * C + 8 * q);
      const bf16x8 al = *reinterpret_cast<const bf16x8*>(sTPL + (16 * mu + r) * C + 8 * q);
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        const bf16x8 bv =
            *reinterpret_cast<const bf16x8*>(sVT + (32 * w + 16 * nt + r) * C + 8 * q);
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        acc = mma(al, bv, acc);
        U[mu][nt] = mma(ah, bv, acc);
      }
    }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      bf16x8 sh[2], slo[2];
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          __bf16 a, b;
          split(S[2 * kk + (e >> 2)][nt][e & 3], a, b);
          sh[nt][e] = a;
          slo[nt][e] = b;
        }
#pragma unroll
      for (int mu = 0; mu < 2; ++mu) {
        const int o = (16 * mu + r) * D + 32 * kk + 4 * q;
        const bf16x8 ah = cat(*reinterpret_cast<const bf16x4*>(sWNH + o),
                              *reinterpret_cast<const bf16x4*>(sWNH + o + 16));
        const bf16x8 al = cat(*reinterpret_cast<const bf16x4*>(sWNL + o),
                              *reinterpret_cast<const bf16x4*>(sWNL + o + 16));
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) U[mu][nt] = mma3(ah, al, sh[nt], slo[nt], U[mu][nt]);
      }
    }

    // ---- S' <- Diag(exp(G_C)) S' + K_H^T U ----------------------------------------------
    bf16x8 uh[2], ul[2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        __bf16 a, b;
        split(U[e >> 2][nt][e & 3], a, b);
        uh[nt][e] = a;
        ul[nt][e] = b;
      }
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) {
      const f32x4 gam = *reinterpret_cast<const f32x4*>(sGam + 16 * mt + 4 * q);
      const int o = (16 * mt + r) * C + 4 * q;
      const bf16x8 ah = cat(*reinterpret_cast<const bf16x4*>(sKHH + o),
                            *reinterpret_cast<const bf16x4*>(sKHH + o + 16));
      const bf16x8 al = cat(*reinterpret_cast<const bf16x4*>(sKHL + o),
                            *reinterpret_cast<const bf16x4*>(sKHL + o + 16));
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        f32x4 s = S[mt][nt] * gam;
        S[mt][nt] = mma3(ah, al, uh[nt], ul[nt], s);
      }
    }
    __syncthreads();
  }

#pragma unroll
  for (int mt = 0; mt < 8; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = 16 * mt + 4 * q + i;
      if (inv_row[head_row + c] < 0) {
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) S_head[int64_t(c) * D + 32 * w + 16 * nt + r] = S[mt][nt][i];
      }
    }
}

}  // namespace

namespace dasc {

bool refresh_wy_supported(int dk, int dv) { return dk == D && dv == D; }

void launch_refresh_wy(bool per_channel, int n_req, int H, int Hqk, int layer, int L,
                       const int32_t* inv_row, float* states, int64_t n_pool, const int32_t* slot,
                       const uint16_t* k, const uint16_t* v, const float* g, const float* beta,
                       int W, int init_zero, hipStream_t st) {
  const dim3 grid(unsigned(n_req) * unsigned(H)), block(256);
  if (per_channel)
    hipLaunchKernelGGL(refresh_wy_kernel<true>, grid, block, 0, st, H, Hqk, layer, L, inv_row,
                       states, n_pool, slot, k, v, g, beta, W, init_zero);
  else
    hipLaunchKernelGGL(refresh_wy_kernel<false>, grid, block, 0, st, H, Hqk, layer, L, inv_row,
                       states, n_pool, slot, k, v, g, beta, W, init_zero);
}

}  // namespace dasc
