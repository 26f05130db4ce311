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
// Software pipeline over chunks (two LDS buffers for a chunk's keys, values, gates and
// A): with b = n mod 2,
//   P1  wave 0 inverts the diagonal blocks of I + A(n); waves 1-3 form X(n) on their
//       columns and stage chunk n+1 into buffer b^1 (wave 1 also sums its gates);
//   P2  wave 0 forms X(n) and one A tile of chunk n+1; wave 1 forms T10(n) and T'(n);
//       waves 2-3 write the rest of T'(n) and the other two A tiles of chunk n+1;
//       waves 1-3 issue the loads of chunk n+2;
//   P3  every wave forms U(n) and updates its columns of S'.
// Three barriers a chunk; the serial inversion runs beside the staging and X.  Register
// chaining, operand splitting, padded LDS rows and the buffer-resource loads (tokens
// past the window read as zeros: identity steps) are as in the channel-wise kernel;
// per-token log-gates are floored at -10 in the same way.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "ckpt_layout.h"
#include "refresh_kernels.h"
#include "wy_ops.h"

namespace {

using namespace dasc_wy;

constexpr int C = 32;       // tokens per chunk
constexpr int D = 128;      // dk = dv
constexpr int DH = 64;      // value columns per block
constexpr float kGateFloor = -10.f;
constexpr float kLog2e = 1.4426950408889634f;

constexpr int SK = 136;     // bf16 [C][SK]   keys, row-major
constexpr int SV = 40;      // bf16 [D][SV]   keys transposed; [DH][SV] values transposed
constexpr int SP = 36;      // bf16 [C][SP]   T'

// LDS map (bytes): one buffer per chunk parity, then T and T' (single).
constexpr int B_K = 0;                          // bf16 [C][SK]  keys
constexpr int B_KT = B_K + C * SK * 2;          // bf16 [D][SV]  keys transposed
constexpr int B_VT = B_KT + D * SV * 2;         // bf16 [DH][SV] this half's values transposed
constexpr int B_A = B_VT + DH * SV * 2;         // f32  [C][C]   A
constexpr int B_G = B_A + C * C * 4;            // f32  [C] G_t
constexpr int B_EG = B_G + C * 4;               // f32  [C] 2^{G_t}
constexpr int B_EH = B_EG + C * 4;              // f32  [C] 2^{G_C - G_t}
constexpr int B_BETA = B_EH + C * 4;            // f32  [C]
constexpr int BUF = B_BETA + C * 4;
constexpr int OFF_T = 2 * BUF;                  // f32  [C][C]
constexpr int OFF_TPH = OFF_T + C * C * 4;      // bf16 [C][SP]
constexpr int OFF_TPL = OFF_TPH + C * SP * 2;
constexpr int LDS_BYTES = OFF_TPL + C * SP * 2;
static_assert(BUF % 16 == 0 && LDS_BYTES <= 81920, "two blocks per CU");

// One DPP move: lane l takes v from the lane CTRL selects within its row of 16 (0 where
// that lane is outside the row); rows outside ROW_MASK keep 0.
template <int CTRL, int ROW_MASK>
__device__ inline float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                               ROW_MASK, 0xF, true));
}

// Inclusive prefix sum over lanes 0..31: shifts by 1, 2, 4, 8 within each row of 16
// lanes, then row 1 adds the last lane of row 0 (row_bcast:15).  No LDS round trips.
__device__ inline float scan32(float x) {
  x += dpp<0x111, 0xF>(x);   // row_shr:1
  x += dpp<0x112, 0xF>(x);   // row_shr:2
  x += dpp<0x114, 0xF>(x);   // row_shr:4
  x += dpp<0x118, 0xF>(x);   // row_shr:8
  x += dpp<0x142, 0xA>(x);   // row_bcast:15 into rows 1 and 3
  return x;
}

// Blocks are dealt to the eight XCDs in turn (block b starts on XCD b mod 8).  Renumber
// them so that each XCD takes a contiguous range of (request, head, half) items: the
// blocks that read one key head (both halves of every v-head in its group) then sit on
// the same XCD and share its L2.  A bijection whenever the grid is a multiple of 8.
__device__ inline int xcd_major(int b, int n_blocks) {
  if (n_blocks & 7) return b;
  return (b & 7) * (n_blocks >> 3) + (b >> 3);
}

// FUSED: the initial state comes from the packed checkpoint (kept rows from their
// packed position, written back to the pool at once; omitted rows +0.0) and every row
// of the layer is written, as the channel-wise kernel's fused variant does.
template <bool FUSED>
__global__ __launch_bounds__(256, 2) void refresh_wy_gdn_kernel(
    int H, int Hqk, int layer, int L, const int32_t* __restrict__ inv_row,
    float* __restrict__ states, int64_t n_pool, const int32_t* __restrict__ slot,
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ v, const float* __restrict__ g,
    const float* __restrict__ beta, int W, int init_zero, dasc::CkptView ck) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[LDS_BYTES];
  float* sT = reinterpret_cast<float*>(smem + OFF_T);
  __bf16* sTPH = reinterpret_cast<__bf16*>(smem + OFF_TPH);
  __bf16* sTPL = reinterpret_cast<__bf16*>(smem + OFF_TPL);
  auto bK = [&](int b) { return reinterpret_cast<uint16_t*>(smem + b * BUF + B_K); };
  auto bKT = [&](int b) { return reinterpret_cast<uint16_t*>(smem + b * BUF + B_KT); };
  auto bVT = [&](int b) { return reinterpret_cast<uint16_t*>(smem + b * BUF + B_VT); };
  auto bA = [&](int b) { return reinterpret_cast<float*>(smem + b * BUF + B_A); };
  auto bG = [&](int b) { return reinterpret_cast<float*>(smem + b * BUF + B_G); };
  auto bEG = [&](int b) { return reinterpret_cast<float*>(smem + b * BUF + B_EG); };
  auto bEH = [&](int b) { return reinterpret_cast<float*>(smem + b * BUF + B_EH); };
  auto bBeta = [&](int b) { return reinterpret_cast<float*>(smem + b * BUF + B_BETA); };

  const int item = xcd_major(blockIdx.x, gridDim.x);
  const int half = item & 1;
  const int nh = item >> 1;
  const int n = nh / H;
  const int h = nh - n * H;
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int q = lane >> 4, r = lane & 15;

  const int64_t head_row = (int64_t(layer) * H + h) * D;
  bool mine = false;
  if (tid < D) mine = inv_row[head_row + tid] < 0;
  const bool any_omitted = __syncthreads_or(mine);
  if (!FUSED && !any_omitted) return;
  const int64_t sl = slot[n];
  if (sl < 0 || sl >= n_pool) return;
  float* S_head = states + (sl * L * H * D + head_row) * D;
  const int col = DH * half + 16 * w + r;   // this lane's value column
  int64_t cslot = 0;
  if (FUSED) {
    cslot = ck.slot[n];
    if (cslot < 0 || cslot >= ck.n_slots) return;
  }
  // Fused: the head's checkpoint row table (float offsets, or dasc::kOmitted /
  // dasc::kNoRow), in buffer 1's A tile, which the pipeline first writes two barriers
  // after the initial state has been read.
  int64_t* sOff = reinterpret_cast<int64_t*>(smem + BUF + B_A);
  static_assert(D * 8 <= C * C * 4, "row table must fit in an A tile");
  if (FUSED) {
    if (tid < D) sOff[tid] = dasc::ckpt_row_offset(inv_row[head_row + tid], ck, cslot, D);
    __syncthreads();
  }
  if (FUSED && !any_omitted) {   // nothing to replay: restore this half of the columns
    for (int e = tid; e < D * DH / 4; e += 256) {
      const int c = e / (DH / 4), v4 = e % (DH / 4);
      const int64_t o = sOff[c];
      const f32x4 val = o >= 0 ? reinterpret_cast<const f32x4*>(ck.ckpt + o + DH * half)[v4]
                               : f32x4{0.f, 0.f, 0.f, 0.f};
      reinterpret_cast<f32x4*>(S_head + int64_t(c) * D + DH * half)[v4] = val;
    }
    return;
  }

  // S'[c][col] for c = 16 mt + 4q + i
  f32x4 S[8];
#pragma unroll
  for (int mt = 0; mt < 8; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = 16 * mt + 4 * q + i;
      if (FUSED) {
        const int64_t o = sOff[c];
        const float val = o >= 0 ? ck.ckpt[o + col] : 0.f;
        S[mt][i] = init_zero ? 0.f : val;
        if (o != dasc::kOmitted) S_head[int64_t(c) * D + col] = val;
      } else {
        S[mt][i] = init_zero ? 0.f : S_head[int64_t(c) * D + col];
      }
    }

  const int hk = h / (H / Hqk);
  const uint16_t* kp = k + (int64_t(n) * Hqk + hk) * W * D;
  const uint16_t* vp = v + (int64_t(n) * H + h) * W * D;
  const float* gp = g + (int64_t(n) * H + h) * W;
  const float* bp = beta + (int64_t(n) * H + h) * W;
  const __amdgpu_buffer_rsrc_t rk = rsrc(kp, W * D * 2), rv = rsrc(vp, W * D * 2);
  const __amdgpu_buffer_rsrc_t rg = rsrc(gp, W * 4), rb = rsrc(bp, W * 4);

  // Waves 1-3 (192 threads, index st = tid - 64) load and stage a chunk:
  //   keys row-major: 8-channel units u = st + 192 i (< 512): token u / 16, channels 8 (u % 16);
  //   keys transposed: items p (< 256): channels 2 (p % 64), +1, tokens 8 (p / 64) .. +7;
  //   values: items p (< 256): columns 64 half + 2 (p % 32), +1, tokens 4 (p / 32) .. +3;
  //     item p = st for every wave and, on wave 3, also 192 + lane (wave 1 sums the gates);
  //   gate and beta: token st % 32 (wave 1 sums them).
  const int st = tid - 64;
  uint4 kraw[3];
  uint32_t kw[2][8], vw[2][4];
  float graw = 0.f, braw = 0.f;
  auto fetch = [&](int c0) {
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      const int u = st + 192 * i;
      if (u < 512)
        kraw[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                                rk, ((u >> 4) * D + (u & 15) * 8) * 2, c0 * D * 2, 0));
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int p = i == 0 ? st : (w == 3 ? 192 + lane : 256);
      if (p < 256) {
#pragma unroll
        for (int j = 0; j < 8; ++j)
          kw[i][j] = __builtin_amdgcn_raw_buffer_load_b32(rk, ((8 * (p >> 6) + j) * D + 2 * (p & 63)) * 2,
                                                          c0 * D * 2, 0);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          vw[i][j] = __builtin_amdgcn_raw_buffer_load_b32(
              rv, ((4 * (p >> 5) + j) * D + DH * half + 2 * (p & 31)) * 2, c0 * D * 2, 0);
      }
    }
    graw = ldf(rg, (st & (C - 1)) * 4, c0 * 4);
    braw = ldf(rb, (st & (C - 1)) * 4, c0 * 4);
  };
  auto stage = [&](int b) {
    uint16_t* sK = bK(b);
    uint16_t* sKT = bKT(b);
    uint16_t* sVT = bVT(b);
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      const int u = st + 192 * i;
      if (u < 512) *reinterpret_cast<uint4*>(sK + (u >> 4) * SK + (u & 15) * 8) = kraw[i];
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int p = i == 0 ? st : (w == 3 ? 192 + lane : 256);
      if (p < 256) {
        uint32_t lo[4], hi[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          lo[j] = __builtin_amdgcn_perm(kw[i][2 * j + 1], kw[i][2 * j], 0x05040100u);
          hi[j] = __builtin_amdgcn_perm(kw[i][2 * j + 1], kw[i][2 * j], 0x07060302u);
        }
        const int c2 = 2 * (p & 63), t8 = 8 * (p >> 6);
        *reinterpret_cast<uint4*>(sKT + c2 * SV + t8) = make_uint4(lo[0], lo[1], lo[2], lo[3]);
        *reinterpret_cast<uint4*>(sKT + (c2 + 1) * SV + t8) = make_uint4(hi[0], hi[1], hi[2], hi[3]);
        const uint32_t vlo0 = __builtin_amdgcn_perm(vw[i][1], vw[i][0], 0x05040100u);
        const uint32_t vlo1 = __builtin_amdgcn_perm(vw[i][3], vw[i][2], 0x05040100u);
        const uint32_t vhi0 = __builtin_amdgcn_perm(vw[i][1], vw[i][0], 0x07060302u);
        const uint32_t vhi1 = __builtin_amdgcn_perm(vw[i][3], vw[i][2], 0x07060302u);
        const int v2 = 2 * (p & 31), t4 = 4 * (p >> 5);
        *reinterpret_cast<uint2*>(sVT + v2 * SV + t4) = make_uint2(vlo0, vlo1);
        *reinterpret_cast<uint2*>(sVT + (v2 + 1) * SV + t4) = make_uint2(vhi0, vhi1);
      }
    }
    if (w == 1) {   // inclusive running sum of the log2 gates over lanes 0..31
      const float x = scan32(lane < C ? fmaxf(graw, kGateFloor) * kLog2e : 0.f);
      const float gc = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), C - 1));
      if (lane < C) {
        bG(b)[lane] = x;
        bEG(b)[lane] = ex2(x);
        bEH(b)[lane] = ex2(gc - x);
        bBeta(b)[lane] = braw;
      }
    }
  };
  // A of the chunk in buffer b, strictly lower, tile (0,0), (1,0) or (1,1)
  auto a_tile = [&](int b, int tile) {
    const uint16_t* sK = bK(b);
    const float* sG = bG(b);
    const float* sBeta = bBeta(b);
    float* sA = bA(b);
    {
      const int ti = tile == 0 ? 0 : 1, si = tile == 2 ? 1 : 0;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const bf16x8 a8 = *reinterpret_cast<const bf16x8*>(sK + (16 * ti + r) * SK + 32 * kk + 8 * q);
        const bf16x8 b8 = *reinterpret_cast<const bf16x8*>(sK + (16 * si + r) * SK + 32 * kk + 8 * q);
        acc = mma(a8, b8, acc);
      }
      const int s = 16 * si + r;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = 16 * ti + 4 * q + i;
        sA[t * C + s] = s < t ? sBeta[t] * acc[i] * ex2(sG[t] - sG[s]) : 0.f;
      }
    }
  };
  // X = Diag(2^G) (K S') on this wave's columns
  auto form_x = [&](int b, f32x4* X) {
    const __bf16* sK = reinterpret_cast<const __bf16*>(bK(b));
    X[0] = f32x4{0.f, 0.f, 0.f, 0.f};
    X[1] = X[0];
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
        const bf16x8 kk8 = ld_op(sK + (16 * mu + r) * SK + 32 * kk + 4 * q);
        X[mu] = mma(kk8, slo, X[mu]);
        X[mu] = mma(kk8, sh, X[mu]);
      }
    }
#pragma unroll
    for (int mu = 0; mu < 2; ++mu) X[mu] *= *reinterpret_cast<const f32x4*>(bEG(b) + 16 * mu + 4 * q);
  };

  // prologue: chunk 0 staged and its A built; chunk 1 in flight
  if (w > 0) fetch(0);
  if (w > 0) stage(0);
  __syncthreads();
  if (w != 1) a_tile(0, w == 0 ? 0 : w - 1);
  if (w > 0) fetch(C);
  __syncthreads();

  for (int t0 = 0, b = 0; t0 < W; t0 += C, b ^= 1) {
    const bool more = t0 + C < W;
    f32x4 X[2];
    // ---- P1: T = (I + A)^{-1} diagonal blocks (wave 0) | X and the next chunk's staging
    if (w == 0) {
      if (lane < 32) {
        const float* sA = bA(b);
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
    } else {
      form_x(b, X);
      if (more) stage(b ^ 1);
    }
    __syncthreads();

    // ---- P2: X (wave 0) | -T' = -T Diag(beta) split (negated so that U takes X - V, one
    //          dot2 per value), T10 = -T11 (A10 T00) on wave 1 |
    //          the next chunk's A tiles (waves 2-3) | loads of the chunk after next
    {
      const float* sA = bA(b);
      const float* sBeta = bBeta(b);
      if (w == 0) {
        form_x(b, X);
        if (more) a_tile(b ^ 1, 0);   // the next chunk's A: tile (0,0) here, the others on waves 2-3
      } else if (w == 1) {
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
          __bf16 a, bb;
          split(z[i] * br, a, bb);   // -T'10
          sTPH[t * SP + r] = a;
          sTPL[t * SP + r] = bb;
        }
      }
      if (w >= 1) {
        // 768 entries outside block (1,0): rows 0..15 whole, rows 16..31 columns 16..31,
        // over waves 1-3 (wave 1 after its T10)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int e = st + 192 * u;
          const int t = e < 512 ? e >> 5 : 16 + ((e - 512) >> 4);
          const int s = e < 512 ? e & 31 : 16 + ((e - 512) & 15);
          const float val = s <= t ? sT[t * C + s] * sBeta[s] : 0.f;
          __bf16 a, bb;
          split(-val, a, bb);
          sTPH[t * SP + s] = a;
          sTPL[t * SP + s] = bb;
        }
        if (w >= 2 && more) a_tile(b ^ 1, w - 1);
        if (t0 + 2 * C < W) fetch(t0 + 2 * C);
      }
    }
    __syncthreads();

    // ---- P3: U = (-T')(X - V), Diag(2^{G_C - G}) U, S' <- 2^{G_C} S' + K^T U ----------
    {
      const uint16_t* sVT = bVT(b);
      const float* sEH = bEH(b);
      f32x4 U[2];
      bf16x8 yh, yl;
      float x[8];
#pragma unroll
      for (int mu = 0; mu < 2; ++mu) {
        const uint2 vv = *reinterpret_cast<const uint2*>(sVT + (16 * w + r) * SV + 16 * mu + 4 * q);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          x[4 * mu + i] = dot2(as_bf2(i < 2 ? vv.x : vv.y), (i & 1) ? kNegHi : kNegLo, X[mu][i]);
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
      bf16x8 uh, ul;
      {
        float xu[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) xu[e] = U[e >> 2][e & 3];
        split8(xu, uh, ul);
      }
      const float gam = bEG(b)[C - 1];
      const __bf16* sKT = reinterpret_cast<const __bf16*>(bKT(b));
#pragma unroll
      for (int mt = 0; mt < 8; ++mt) {
        const bf16x8 kt8 = ld_op(sKT + (16 * mt + r) * SV + 4 * q);
        S[mt] = mma(kt8, ul, S[mt] * gam);
        S[mt] = mma(kt8, uh, S[mt]);
      }
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
  const CkptView none{nullptr, 1, 1, 0, nullptr};
  hipLaunchKernelGGL(refresh_wy_gdn_kernel<false>, grid, block, 0, st, H, Hqk, layer, L, inv_row,
                     states, n_pool, slot, k, v, g, beta, W, init_zero, none);
}

void launch_restore_refresh_wy_gdn(int n_req, int H, int Hqk, int layer, int L, const float* ckpt,
                                   int64_t n_ckpt_slots, const int32_t* ck_slot,
                                   int64_t slice_rows, int64_t n_rows, const int32_t* inv_row,
                                   float* states, int64_t n_pool, const int32_t* slot,
                                   const uint16_t* k, const uint16_t* v, const float* g,
                                   const float* beta, int W, int init_zero, hipStream_t st) {
  const dim3 grid(unsigned(n_req) * unsigned(H) * 2u), block(256);
  const CkptView ck{ckpt, n_ckpt_slots, slice_rows, n_rows, ck_slot};
  hipLaunchKernelGGL(refresh_wy_gdn_kernel<true>, grid, block, 0, st, H, Hqk, layer, L, inv_row,
                     states, n_pool, slot, k, v, g, beta, W, init_zero, ck);
}

}  // namespace dasc
