// Chunkwise WY-form refresh for GDN heads (one scalar gate per token), dk = dv = 128,
// on bf16 MFMA (gfx950).
//
// Same recurrence and chunk algebra as the channel-wise kernel (Sec. 3.1, Eq. 1 on
// S' = S^T, chunks of C = 32 tokens, G_t = sum_{r<=t} g_r in log2 units), but with a
// scalar decay per token every decay factor leaves the contractions:
//     A_ts = beta_t (K K^T)_ts 2^{G_t - G_s}           (s < t)
//     X    = K_G S' = Diag(2^{G_t}) (K S')
//     S'  <- 2^{G_C} S' + K^T (Diag(2^{G_C - G_t}) U),  U = T'(V - X)
// Keys are bf16, so K is an exact MFMA operand: K K^T takes one bf16 pass (the products
// are exact in fp32) and K S', K^T U take two (state and update split into bf16 hi + lo)
// instead of three.  Only 32 exponentials per chunk remain, and no K_G / K_H tiles are
// built.
//
// Work split: one 256-thread block per (request, head, half of the value columns); wave
// w owns columns [64 half + 16 w, +16) of S' (128 x 16 fp32 in MFMA accumulators).  The
// S-independent part (A, T, T') is recomputed by both halves; it is cheap here, and the
// split doubles the blocks of a launch (a layer of a GDN model has few omitted heads).
//
// Per chunk: stage (keys row-major and transposed, this half's values transposed, gates
// and beta; the running sum of the gates on wave 0) | A tiles on waves 0-2 and X on
// every wave | T = (I + A)^{-1} diagonal blocks on wave 0 | T' (T10 on wave 1) | U and
// the state update.  Register chaining, operand splitting, padded LDS rows and the
// buffer-resource loads (tokens past the window read as zeros: identity steps) are as
// in the channel-wise kernel; per-token log-gates are floored at -10 in the same way.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "refresh_kernels.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int C = 32;       // tokens per chunk
constexpr int D = 128;      // dk = dv
constexpr int DH = 64;      // value columns per block
constexpr float kGateFloor = -10.f;
constexpr float kLog2e = 1.4426950408889634f;

constexpr int SK = 136;     // bf16 [C][SK]   keys, row-major
constexpr int SV = 40;      // bf16 [D][SV]   keys transposed; [DH][SV] values transposed
constexpr int SP = 36;      // bf16 [C][SP]   T'

constexpr int OFF_K = 0;                        // bf16 [C][SK]
constexpr int OFF_KT = OFF_K + C * SK * 2;      // bf16 [D][SV]
constexpr int OFF_VT = OFF_KT + D * SV * 2;     // bf16 [DH][SV]
constexpr int OFF_A = OFF_VT + DH * SV * 2;     // f32  [C][C]
constexpr int OFF_T = OFF_A + C * C * 4;        // f32  [C][C]
constexpr int OFF_TPH = OFF_T + C * C * 4;      // bf16 [C][SP]
constexpr int OFF_TPL = OFF_TPH + C * SP * 2;
constexpr int OFF_G = OFF_TPL + C * SP * 2;     // f32  [C] G_t
constexpr int OFF_EG = OFF_G + C * 4;           // f32  [C] 2^{G_t}
constexpr int OFF_EH = OFF_EG + C * 4;          // f32  [C] 2^{G_C - G_t}
constexpr int OFF_BETA = OFF_EH + C * 4;        // f32  [C]
constexpr int LDS_BYTES = OFF_BETA + C * 4;

__device__ inline float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ inline __amdgpu_buffer_rsrc_t rsrc(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes, 0x00020000);
}
__device__ inline float ldf(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}

__device__ inline void split(float x, __bf16& hi, __bf16& lo) {
  hi = static_cast<__bf16>(x);
  lo = static_cast<__bf16>(x - static_cast<float>(hi));
}

// Eight values split at once: two values per packed conversion.
__device__ inline void split8(const float* x, bf16x8& hi, bf16x8& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const uint32_t hw = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{x[2 * p], x[2 * p + 1]}, bf16x2));
    const float r0 = __uint_as_float(hw << 16), r1 = __uint_as_float(hw & 0xFFFF0000u);
    h[p] = hw;
    l[p] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{x[2 * p] - r0, x[2 * p + 1] - r1}, bf16x2));
  }
  hi = __builtin_bit_cast(bf16x8, make_uint4(h[0], h[1], h[2], h[3]));
  lo = __builtin_bit_cast(bf16x8, make_uint4(l[0], l[1], l[2], l[3]));
}

__device__ inline f32x4 mma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ inline f32x4 mma32(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ inline bf16x8 cat(bf16x4 a, bf16x4 b) {
  return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// Row-major bf16 operand with the contraction index k(q, e) (four values at p, four at
// p + 16).
__device__ inline bf16x8 ld_op(const __bf16* p) {
  return cat(*reinterpret_cast<const bf16x4*>(p), *reinterpret_cast<const bf16x4*>(p + 16));
}

__global__ __launch_bounds__(256, 2) void refresh_wy_gdn_kernel(
    int H, int Hqk, int layer, int L, const int32_t* __restrict__ inv_row,
    float* __restrict__ states, int64_t n_pool, const int32_t* __restrict__ slot,
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ v, const float* __restrict__ g,
    const float* __restrict__ beta, int W, int init_zero) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[LDS_BYTES];
  uint16_t* sK = reinterpret_cast<uint16_t*>(smem + OFF_K);
  uint16_t* sKT = reinterpret_cast<uint16_t*>(smem + OFF_KT);
  uint16_t* sVT = reinterpret_cast<uint16_t*>(smem + OFF_VT);
  float* sA = reinterpret_cast<float*>(smem + OFF_A);
  float* sT = reinterpret_cast<float*>(smem + OFF_T);
  __bf16* sTPH = reinterpret_cast<__bf16*>(smem + OFF_TPH);
  __bf16* sTPL = reinterpret_cast<__bf16*>(smem + OFF_TPL);
  float* sG = reinterpret_cast<float*>(smem + OFF_G);
  float* sEG = reinterpret_cast<float*>(smem + OFF_EG);
  float* sEH = reinterpret_cast<float*>(smem + OFF_EH);
  float* sBeta = reinterpret_cast<float*>(smem + OFF_BETA);

  const int half = blockIdx.x & 1;
  const int nh = blockIdx.x >> 1;
  const int n = nh / H;
  const int h = nh - n * H;
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
  const int col = DH * half + 16 * w + r;   // this lane's value column

  // S'[c][col] for c = 16 mt + 4q + i
  f32x4 S[8];
#pragma unroll
  for (int mt = 0; mt < 8; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      S[mt][i] = init_zero ? 0.f : S_head[int64_t(16 * mt + 4 * q + i) * D + col];

  const int hk = h / (H / Hqk);
  const uint16_t* kp = k + (int64_t(n) * Hqk + hk) * W * D;
  const uint16_t* vp = v + (int64_t(n) * H + h) * W * D;
  const float* gp = g + (int64_t(n) * H + h) * W;
  const float* bp = beta + (int64_t(n) * H + h) * W;
  const __amdgpu_buffer_rsrc_t rk = rsrc(kp, W * D * 2), rv = rsrc(vp, W * D * 2);
  const __amdgpu_buffer_rsrc_t rg = rsrc(gp, W * 4), rb = rsrc(bp, W * 4);

  // Load ownership (issued one chunk ahead):
  //   keys row-major: two 8-channel units (token kt, channels kc8..) per thread;
  //   keys transposed: channels 2p, 2p + 1 of tokens 8o .. 8o+7 (p = tid % 64, o = tid / 64);
  //   values: columns 64 half + 2p', +1 of tokens 4o' .. 4o'+3 (p' = tid % 32, o' = tid / 32);
  //   gate and beta: token tid (threads below 32).
  const int kp2 = tid & 63, ko = tid >> 6;
  const int vp2 = tid & 31, vo = tid >> 5;
  uint4 kraw[2];
  uint32_t kw[8], vw[4];
  float graw, braw;
  auto fetch = [&](int c0) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int t = (tid + 256 * u) >> 4, c8 = ((tid + 256 * u) & 15) * 8;
      kraw[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rk, (t * D + c8) * 2, c0 * D * 2, 0));
    }
#pragma unroll
    for (int i = 0; i < 8; ++i)
      kw[i] = __builtin_amdgcn_raw_buffer_load_b32(rk, ((8 * ko + i) * D + 2 * kp2) * 2, c0 * D * 2, 0);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      vw[i] = __builtin_amdgcn_raw_buffer_load_b32(rv, ((4 * vo + i) * D + DH * half + 2 * vp2) * 2,
                                                   c0 * D * 2, 0);
    graw = ldf(rg, (tid & (C - 1)) * 4, c0 * 4);
    braw = ldf(rb, (tid & (C - 1)) * 4, c0 * 4);
  };
  fetch(0);

  for (int t0 = 0; t0 < W; t0 += C) {
    // ---- stage: keys (both layouts), this half's values, beta, the gates' running sum
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int t = (tid + 256 * u) >> 4, c8 = ((tid + 256 * u) & 15) * 8;
      *reinterpret_cast<uint4*>(sK + t * SK + c8) = kraw[u];
    }
    {
      uint32_t lo[4], hi[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        lo[i] = __builtin_amdgcn_perm(kw[2 * i + 1], kw[2 * i], 0x05040100u);
        hi[i] = __builtin_amdgcn_perm(kw[2 * i + 1], kw[2 * i], 0x07060302u);
      }
      *reinterpret_cast<uint4*>(sKT + (2 * kp2) * SV + 8 * ko) = make_uint4(lo[0], lo[1], lo[2], lo[3]);
      *reinterpret_cast<uint4*>(sKT + (2 * kp2 + 1) * SV + 8 * ko) = make_uint4(hi[0], hi[1], hi[2], hi[3]);
    }
    {
      const uint32_t lo0 = __builtin_amdgcn_perm(vw[1], vw[0], 0x05040100u);
      const uint32_t lo1 = __builtin_amdgcn_perm(vw[3], vw[2], 0x05040100u);
      const uint32_t hi0 = __builtin_amdgcn_perm(vw[1], vw[0], 0x07060302u);
      const uint32_t hi1 = __builtin_amdgcn_perm(vw[3], vw[2], 0x07060302u);
      *reinterpret_cast<uint2*>(sVT + (2 * vp2) * SV + 4 * vo) = make_uint2(lo0, lo1);
      *reinterpret_cast<uint2*>(sVT + (2 * vp2 + 1) * SV + 4 * vo) = make_uint2(hi0, hi1);
    }
    if (w == 0) {   // inclusive running sum over the 32 tokens by lane shuffles
      float x = lane < C ? fmaxf(graw, kGateFloor) * kLog2e : 0.f;
#pragma unroll
      for (int d = 1; d < C; d <<= 1) {
        const float y = __shfl_up(x, d);
        if (lane >= d) x += y;
      }
      const float gc = __shfl(x, C - 1);
      if (lane < C) {
        sG[lane] = x;
        sEG[lane] = ex2(x);
        sEH[lane] = ex2(gc - x);
        sBeta[lane] = braw;
      }
    }
    __syncthreads();

    // ---- A = Diag(beta) (K K^T with decays), strictly lower: waves 0-2, one tile each;
    // X = Diag(2^G) (K S') on every wave's own columns
    if (w < 3) {
      const int ti = w == 0 ? 0 : 1, si = w == 2 ? 1 : 0;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(sK + (16 * ti + r) * SK + 32 * kk + 8 * q);
        const bf16x8 b = *reinterpret_cast<const bf16x8*>(sK + (16 * si + r) * SK + 32 * kk + 8 * q);
        acc = mma(a, b, acc);
      }
      const int s = 16 * si + r;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = 16 * ti + 4 * q + i;
        sA[t * C + s] = s < t ? sBeta[t] * acc[i] * ex2(sG[t] - sG[s]) : 0.f;
      }
    }
    f32x4 X[2] = {};
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      bf16x8 sh, slo;
      {
        float x[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = S[2 * kk + (e >> 2)][e & 3];
        split8(x, sh, slo);
      }
#pragma unroll
      for (int mu = 0; mu < 2; ++mu) {
        const bf16x8 kk8 = ld_op(reinterpret_cast<const __bf16*>(sK) + (16 * mu + r) * SK + 32 * kk + 4 * q);
        X[mu] = mma(kk8, slo, X[mu]);
        X[mu] = mma(kk8, sh, X[mu]);
      }
    }
#pragma unroll
    for (int mu = 0; mu < 2; ++mu) {
      const f32x4 eg = *reinterpret_cast<const f32x4*>(sEG + 16 * mu + 4 * q);
      X[mu] *= eg;
    }
    __syncthreads();

    // ---- T = (I + A)^{-1}: diagonal 16x16 blocks by forward substitution -----------
    if (w == 0 && lane < 32) {
      const int base = 16 * (lane >> 4), s = lane & 15;
      float x[16];
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        float a = (t == s) ? 1.f : 0.f;
#pragma unroll
        for (int rr = 0; rr < t; ++rr) a = fmaf(-sA[(base + t) * C + base + rr], x[rr], a);
        x[t] = a;
        sT[(base + t) * C + base + s] = a;
      }
    }
    // the next chunk's inputs load while this chunk finishes (zeros past the window)
    fetch(t0 + C);
    __syncthreads();

    // ---- T' = T Diag(beta), split hi/lo; wave 1 forms T10 = -T11 (A10 T00) ---------
    if (w == 1) {
      f32x4 y = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < 4; ++i)
        y = mma32(sA[(16 + r) * C + 4 * q + i], sT[(4 * q + i) * C + r], y);
      f32x4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < 4; ++i) z = mma32(sT[(16 + r) * C + 16 + 4 * q + i], y[i], z);
      const float br = sBeta[r];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = 16 + 4 * q + i;
        __bf16 a, b;
        split(-z[i] * br, a, b);
        sTPH[t * SP + r] = a;
        sTPL[t * SP + r] = b;
      }
    } else {
      const int lt = w == 0 ? tid : tid - 64;       // 0 .. 191
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        // 768 entries outside block (1,0): rows 0..15 whole, rows 16..31 columns 16..31
        const int e = lt + 192 * u;
        const int t = e < 512 ? e >> 5 : 16 + ((e - 512) >> 4);
        const int s = e < 512 ? e & 31 : 16 + ((e - 512) & 15);
        const float val = s <= t ? sT[t * C + s] * sBeta[s] : 0.f;
        __bf16 a, b;
        split(val, a, b);
        sTPH[t * SP + s] = a;
        sTPL[t * SP + s] = b;
      }
    }
    __syncthreads();

    // ---- U = T' (V - X), then Diag(2^{G_C - G}) U -----------------------------------
    f32x4 U[2];
    {
      bf16x8 yh, yl;
      float x[8];
#pragma unroll
      for (int mu = 0; mu < 2; ++mu) {
        const uint2 vv = *reinterpret_cast<const uint2*>(sVT + (16 * w + r) * SV + 16 * mu + 4 * q);
        const float vf[4] = {__uint_as_float(vv.x << 16), __uint_as_float(vv.x & 0xFFFF0000u),
                             __uint_as_float(vv.y << 16), __uint_as_float(vv.y & 0xFFFF0000u)};
#pragma unroll
        for (int i = 0; i < 4; ++i) x[4 * mu + i] = vf[i] - X[mu][i];
      }
      split8(x, yh, yl);
#pragma unroll
      for (int mu = 0; mu < 2; ++mu) {
        const int o = (16 * mu + r) * SP + 4 * q;
        const bf16x8 ah = ld_op(sTPH + o), al = ld_op(sTPL + o);
        f32x4 c = mma(al, yh, f32x4{0.f, 0.f, 0.f, 0.f});
        c = mma(ah, yl, c);
        U[mu] = mma(ah, yh, c);
        U[mu] *= *reinterpret_cast<const f32x4*>(sEH + 16 * mu + 4 * q);
      }
    }

    // ---- S' <- 2^{G_C} S' + K^T U -----------------------------------------------------
    bf16x8 uh, ul;
    {
      float x[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = U[e >> 2][e & 3];
      split8(x, uh, ul);
    }
    const float gam = sEG[C - 1];
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) {
      const bf16x8 kt8 = ld_op(reinterpret_cast<const __bf16*>(sKT) + (16 * mt + r) * SV + 4 * q);
      S[mt] = mma(kt8, ul, S[mt] * gam);
      S[mt] = mma(kt8, uh, S[mt]);
    }
    __syncthreads();
  }

#pragma unroll
  for (int mt = 0; mt < 8; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = 16 * mt + 4 * q + i;
      if (inv_row[head_row + c] < 0) S_head[int64_t(c) * D + col] = S[mt][i];
    }
}

}  // namespace

namespace dasc {

void launch_refresh_wy_gdn(int n_req, int H, int Hqk, int layer, int L, const int32_t* inv_row,
                           float* states, int64_t n_pool, const int32_t* slot, const uint16_t* k,
                           const uint16_t* v, const float* g, const float* beta, int W,
                           int init_zero, hipStream_t st) {
  const dim3 grid(unsigned(n_req) * unsigned(H) * 2u), block(256);
  hipLaunchKernelGGL(refresh_wy_gdn_kernel, grid, block, 0, st, H, Hqk, layer, L, inv_row, states,
                     n_pool, slot, k, v, g, beta, W, init_zero);
}

}  // namespace dasc
