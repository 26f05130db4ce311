// Chunkwise WY-form refresh for GDN heads (one scalar gate per token), dk = dv = 128,
// on bf16 MFMA (gfx950), in two launches.
//
// Same recurrence and chunk algebra as the channel-wise kernel (Sec. 3.1, Eq. 1 on
// S' = S^T, chunks of C = 32 tokens, G_t = sum_{r<=t} g_r in log2 units), but with a
// scalar decay per token every decay factor leaves the contractions:
//     A_ts = beta_t (K K^T)_ts 2^{G_t - G_s}           (s < t)
//     T'   = (I + A)^{-1} Diag(beta)
//     X    = K_G S' = Diag(2^{G_t}) (K S')
//     S'  <- 2^{G_C} S' + K^T (Diag(2^{G_C - G_t}) U),  U = T'(V - X)
// Keys are bf16, so K is an exact MFMA operand: K K^T takes one bf16 pass (the products
// are exact in fp32) and K S', K^T U take two (state and update split into bf16 hi + lo)
// instead of three.
//
// A and T' do not depend on the state.  gdn_factor_kernel builds them for every chunk
// of every refreshed head at once (one wave per chunk) and stores -T', split into bf16
// hi + lo in the order the U contraction loads it, in the caller's workspace.  The
// state recurrence, refresh_wy_gdn_kernel, then carries per chunk only X, U and the
// update: its serial chain no longer holds the triangular solve, and it takes one
// barrier a chunk.
//
// Recurrence work split: one 256-thread block per (request, head, half of the value
// columns); wave w owns columns [64 half + 16 w, +16) of S' (128 x 16 fp32 in MFMA
// accumulators).  Two LDS buffers alternate by chunk: while a chunk is contracted out of
// one, the next is staged into the other from registers loaded a chunk earlier.
// Register chaining, operand splitting, padded LDS rows and the buffer-resource loads
// (tokens past the window read as zeros: identity steps) are as in the channel-wise
// kernel; per-token log-gates are floored at -10 in the same way.

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

// -T' of one chunk in the workspace: [mu][hi/lo][lane][8 bf16], where lane (q, r) holds
// row 16 mu + r at the register-chained contraction index k(q, e) -- one 16-byte load
// per (mu, hi/lo) and lane.
constexpr int TP_VEC = 2 * 2 * 64;   // uint4 per chunk (4 KiB)
static_assert(TP_VEC * 16 == dasc::kGdnFactorBytesPerChunk, "factor size");

// ---- factor kernel: per-wave LDS (padded f32 rows) ---------------------------------------
// One tile holds A and then, in place, T = (I + A)^{-1}: the substitution overwrites the
// diagonal blocks row by row after reading them, and T10 replaces A10 once A10 T00 is in
// registers.
constexpr int SA = 33;
constexpr int F_M = 0;                       // f32 [C][SA]  A, then T
constexpr int F_G = F_M + C * SA * 4;        // f32 [C]      G_t
constexpr int F_B = F_G + C * 4;             // f32 [C]      beta_t
constexpr int F_WAVE = F_B + C * 4;

// ---- recurrence kernel: LDS, two buffers by chunk parity ---------------------------------
constexpr int SK = 136;     // bf16 [C][SK]   keys, row-major
constexpr int SV = 40;      // bf16 [D][SV]   keys transposed; [DH][SV] values transposed
constexpr int B_K = 0;                          // bf16 [C][SK]  keys, channels interleaved (ilv)
constexpr int B_KT = B_K + C * SK * 2;          // bf16 [D][SV]  keys transposed, tokens interleaved
constexpr int B_VT = B_KT + D * SV * 2;         // bf16 [DH][SV] this half's values transposed, tokens interleaved
constexpr int B_EG = B_VT + DH * SV * 2;        // f32  [C] 2^{G_t}
constexpr int B_EH = B_EG + C * 4;              // f32  [C] 2^{G_C - G_t}
constexpr int BUF = B_EH + C * 4;
constexpr int OFF_ROWS = 2 * BUF;               // int64 [D] fused: checkpoint row table
constexpr int LDS_BYTES = OFF_ROWS + D * 8;
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

// Cumulative log2-decay of a chunk: lane t < 32 ends with G_t (lanes 32..63 hold sums
// of zeros and are not used).
__device__ inline float chunk_log2_decay(float graw, int lane) {
  return scan32(lane < C ? fmaxf(graw, kGateFloor) * kLog2e : 0.f);
}

// Does head h of layer `layer` have an omitted row?  Every thread of the block must call
// it (it is a block barrier).
__device__ inline bool head_refreshed(const int32_t* inv_row, int64_t head_row, int tid) {
  bool mine = false;
  if (tid < D) mine = inv_row[head_row + tid] < 0;
  return __syncthreads_or(mine);
}

// Blocks are dealt to the eight XCDs in turn (block b starts on XCD b mod 8).  Renumber
// them so that each XCD takes a contiguous range of (request, head, half) items: the
// blocks that read one key head (both halves of every v-head in its group) then sit on
// the same XCD and share its L2.  A bijection whenever the grid is a multiple of 8.
__device__ inline int xcd_major(int b, int n_blocks) {
  if (n_blocks & 7) return b;
  return (b & 7) * (n_blocks >> 3) + (b >> 3);
}

// ---------------------------------------------------------------------------------------
// -T' for chunk c of (request n, head h): wave w of block (n H + h) * per_head + j takes
// chunk 4 j + w.  Heads with no omitted row are skipped.  The waves of a block share
// nothing after the first barrier.
__global__ __launch_bounds__(256) void gdn_factor_kernel(
    int H, int Hqk, int layer, const int32_t* __restrict__ inv_row, const uint16_t* __restrict__ k,
    const float* __restrict__ g, const float* __restrict__ beta, int W, int n_chunks,
    uint4* __restrict__ ws) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[4 * F_WAVE];
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int q = lane >> 4, r = lane & 15;
  const int per_head = (n_chunks + 3) >> 2;
  const int nh = blockIdx.x / per_head;
  const int c = 4 * (blockIdx.x - nh * per_head) + w;
  const int n = nh / H, h = nh - n * H;
  if (!head_refreshed(inv_row, (int64_t(layer) * H + h) * D, tid)) return;
  if (c >= n_chunks) return;   // a whole wave past the last chunk

  float* sM = reinterpret_cast<float*>(smem + w * F_WAVE + F_M);
  float* sG = reinterpret_cast<float*>(smem + w * F_WAVE + F_G);
  float* sB = reinterpret_cast<float*>(smem + w * F_WAVE + F_B);

  const int hk = h / (H / Hqk);
  const __amdgpu_buffer_rsrc_t rk = rsrc(k + (int64_t(n) * Hqk + hk) * W * D, W * D * 2);
  const __amdgpu_buffer_rsrc_t rg = rsrc(g + (int64_t(n) * H + h) * W, W * 4);
  const __amdgpu_buffer_rsrc_t rb = rsrc(beta + (int64_t(n) * H + h) * W, W * 4);

  // K K^T, three 16x16 tiles: lane (q, r) loads rows r and 16 + r at channels
  // 32 kk + 8 q .. + 7, which are its A fragment for one tile and its B fragment for
  // another (B[k][n] = K[n][k]).
  bf16x8 f[2][4];
#pragma unroll
  for (int ti = 0; ti < 2; ++ti)
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      f[ti][kk] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(
                                                 rk, ((16 * ti + r) * D + 32 * kk + 8 * q) * 2,
                                                 c * C * D * 2, 0));
  const float graw = lane < C ? ldf(rg, lane * 4, c * C * 4) : 0.f;
  const float braw = lane < C ? ldf(rb, lane * 4, c * C * 4) : 0.f;
  const float G = chunk_log2_decay(graw, lane);
  if (lane < C) {
    sG[lane] = G;
    sB[lane] = braw;
  }
  f32x4 acc[3];
#pragma unroll
  for (int tile = 0; tile < 3; ++tile) {
    const int ti = tile == 0 ? 0 : 1, si = tile == 2 ? 1 : 0;
    acc[tile] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) acc[tile] = mma(f[ti][kk], f[si][kk], acc[tile]);
  }
  wave_lds_sync();
  // A = Diag(beta) (strictly lower part of K K^T scaled by 2^{G_t - G_s})
#pragma unroll
  for (int tile = 0; tile < 3; ++tile) {
    const int ti = tile == 0 ? 0 : 1, si = tile == 2 ? 1 : 0;
    const int s = 16 * si + r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = 16 * ti + 4 * q + i;
      sM[t * SA + s] = s < t ? sB[t] * acc[tile][i] * ex2(sG[t] - sG[s]) : 0.f;
    }
  }
  wave_lds_sync();

  // T = (I + A)^{-1}: diagonal 16x16 blocks by forward substitution, lane = column;
  // row t of T replaces row t of A once every lane has read it (the wave runs in step)
  if (lane < 32) {
    const int base = 16 * (lane >> 4), s = lane & 15;
    float x[16];
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      float a = (t == s) ? 1.f : 0.f;
#pragma unroll
      for (int rr = 0; rr < t; ++rr) a = fmaf(-sM[(base + t) * SA + base + rr], x[rr], a);
      x[t] = a;
      sM[(base + t) * SA + base + s] = a;
    }
  }
  wave_lds_sync();

  // T10 = -T11 (A10 T00) on fp32 MFMA, the product staying in registers between the
  // steps; it then takes A10's place
  {
    f32x4 y = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 4; ++i) y = mma32(sM[(16 + r) * SA + 4 * q + i], sM[(4 * q + i) * SA + r], y);
    f32x4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 4; ++i) z = mma32(sM[(16 + r) * SA + 16 + 4 * q + i], y[i], z);
    wave_lds_sync();   // every lane's reads of A10 are done
#pragma unroll
    for (int i = 0; i < 4; ++i) sM[(16 + 4 * q + i) * SA + r] = -z[i];
  }
  wave_lds_sync();

  // -T' = -T Diag(beta) in the U contraction's operand order, split hi/lo
  uint4* out = ws + ((int64_t(n) * H + h) * n_chunks + c) * TP_VEC;
#pragma unroll
  for (int mu = 0; mu < 2; ++mu) {
    const int t = 16 * mu + r;
    float x[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int s = e < 4 ? 4 * q + e : 16 + 4 * q + e - 4;
      x[e] = s <= t ? -(sM[t * SA + s] * sB[s]) : 0.f;
    }
    bf16x8 hi, lo;
    split8(x, hi, lo);
    out[(2 * mu) * 64 + lane] = __builtin_bit_cast(uint4, hi);
    out[(2 * mu + 1) * 64 + lane] = __builtin_bit_cast(uint4, lo);
  }
}

// ---------------------------------------------------------------------------------------
// The state recurrence over the window, -T' of every chunk read from the workspace.
// FUSED: the initial state comes from the packed checkpoint (kept rows from their packed
// position, written back to the pool at once; omitted rows +0.0) and every row of the
// layer is written, as the channel-wise kernel's fused variant does.
template <bool FUSED>
__global__ __launch_bounds__(256, 2) void refresh_wy_gdn_kernel(
    int H, int Hqk, int layer, int L, const int32_t* __restrict__ inv_row,
    float* __restrict__ states, int64_t n_pool, const int32_t* __restrict__ slot,
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ v, const float* __restrict__ g,
    int W, int init_zero, dasc::CkptView ck, const uint4* __restrict__ ws, int n_chunks) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[LDS_BYTES];
  auto bK = [&](int b) { return reinterpret_cast<uint16_t*>(smem + b * BUF + B_K); };
  auto bKT = [&](int b) { return reinterpret_cast<uint16_t*>(smem + b * BUF + B_KT); };
  auto bVT = [&](int b) { return reinterpret_cast<uint16_t*>(smem + b * BUF + B_VT); };
  auto bEG = [&](int b) { return reinterpret_cast<float*>(smem + b * BUF + B_EG); };
  auto bEH = [&](int b) { return reinterpret_cast<float*>(smem + b * BUF + B_EH); };

  const int item = xcd_major(blockIdx.x, gridDim.x);
  const int half = item & 1;
  const int nh = item >> 1;
  const int n = nh / H;
  const int h = nh - n * H;
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int q = lane >> 4, r = lane & 15;

  const int64_t head_row = (int64_t(layer) * H + h) * D;
  const bool any_omitted = head_refreshed(inv_row, head_row, tid);
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
  // dasc::kNoRow).
  int64_t* sOff = reinterpret_cast<int64_t*>(smem + OFF_ROWS);
  if (FUSED) {
    if (tid < D) sOff[tid] = dasc::ckpt_row_offset(inv_row[head_row + tid], ck, cslot, D);
    __syncthreads();
  }
  if (FUSED) {
    // Rows that are not replayed (this half of their columns) are final already: copied
    // from the checkpoint (or +0.0) in one 16-byte-per-thread pass, whose stores drain
    // while the replay runs.  A head with no omitted row is done after this.
    for (int e = tid; e < D * DH / 4; e += 256) {
      const int c = e / (DH / 4), v4 = e % (DH / 4);
      const int64_t o = sOff[c];
      if (!any_omitted || o != dasc::kOmitted) {
        const f32x4 val = o >= 0 ? reinterpret_cast<const f32x4*>(ck.ckpt + o + DH * half)[v4]
                                 : f32x4{0.f, 0.f, 0.f, 0.f};
        reinterpret_cast<f32x4*>(S_head + int64_t(c) * D + DH * half)[v4] = val;
      }
    }
    if (!any_omitted) return;
  }

  // S'[c][col] for c = 16 mt + 4q + i
  f32x4 S[8];
#pragma unroll
  for (int mt = 0; mt < 8; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = 16 * mt + 4 * q + i;
      float val = 0.f;
      if (FUSED) {
        const int64_t o = sOff[c];   // the restored value: kept row, or +0.0
        if (!init_zero && o >= 0) val = ck.ckpt[o + col];
      } else if (!init_zero) {
        val = S_head[int64_t(c) * D + col];
      }
      S[mt][i] = val;
    }

  const int hk = h / (H / Hqk);
  const uint16_t* kp = k + (int64_t(n) * Hqk + hk) * W * D;
  const uint16_t* vp = v + (int64_t(n) * H + h) * W * D;
  const float* gp = g + (int64_t(n) * H + h) * W;
  const __amdgpu_buffer_rsrc_t rk = rsrc(kp, W * D * 2), rv = rsrc(vp, W * D * 2);
  const __amdgpu_buffer_rsrc_t rg = rsrc(gp, W * 4);
  const uint4* tp = ws + (int64_t(n) * H + h) * n_chunks * TP_VEC;

  // Each thread loads and stages a chunk's
  //   keys row-major: 8-channel units u = tid and 256 + tid: token u / 16, channels 8 (u % 16);
  //   keys transposed: channels 2 (tid % 64), +1 at tokens 8 (tid / 64) .. +7;
  //   values: columns 64 half + 2 (tid % 32), +1 at tokens 4 (tid / 32) .. +3;
  // and lanes 0..31 of wave 0 its gates (summed there).
  uint4 kraw[2];
  uint32_t kw[8], vw[4];
  float graw = 0.f;
  auto fetch = [&](int c0) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int u = tid + 256 * i;
      kraw[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                              rk, ((u >> 4) * D + (u & 15) * 8) * 2, c0 * D * 2, 0));
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
      kw[j] = __builtin_amdgcn_raw_buffer_load_b32(rk, ((8 * (tid >> 6) + j) * D + 2 * (tid & 63)) * 2,
                                                   c0 * D * 2, 0);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      vw[j] = __builtin_amdgcn_raw_buffer_load_b32(
          rv, ((4 * (tid >> 5) + j) * D + DH * half + 2 * (tid & 31)) * 2, c0 * D * 2, 0);
    if (w == 0) graw = ldf(rg, (lane & (C - 1)) * 4, c0 * 4);
  };
  auto stage = [&](int b) {
    uint16_t* sK = bK(b);
    uint16_t* sKT = bKT(b);
    uint16_t* sVT = bVT(b);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int u = tid + 256 * i;
      const int c8 = (u & 15) * 8;
      *reinterpret_cast<uint2*>(sK + (u >> 4) * SK + ilv(c8)) = make_uint2(kraw[i].x, kraw[i].y);
      *reinterpret_cast<uint2*>(sK + (u >> 4) * SK + ilv(c8 + 4)) = make_uint2(kraw[i].z, kraw[i].w);
    }
    {
      uint32_t lo[4], hi[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        lo[j] = __builtin_amdgcn_perm(kw[2 * j + 1], kw[2 * j], 0x05040100u);
        hi[j] = __builtin_amdgcn_perm(kw[2 * j + 1], kw[2 * j], 0x07060302u);
      }
      const int c2 = 2 * (tid & 63), t8 = 8 * (tid >> 6);
      *reinterpret_cast<uint2*>(sKT + c2 * SV + ilv(t8)) = make_uint2(lo[0], lo[1]);
      *reinterpret_cast<uint2*>(sKT + c2 * SV + ilv(t8 + 4)) = make_uint2(lo[2], lo[3]);
      *reinterpret_cast<uint2*>(sKT + (c2 + 1) * SV + ilv(t8)) = make_uint2(hi[0], hi[1]);
      *reinterpret_cast<uint2*>(sKT + (c2 + 1) * SV + ilv(t8 + 4)) = make_uint2(hi[2], hi[3]);
      const uint32_t vlo0 = __builtin_amdgcn_perm(vw[1], vw[0], 0x05040100u);
      const uint32_t vlo1 = __builtin_amdgcn_perm(vw[3], vw[2], 0x05040100u);
      const uint32_t vhi0 = __builtin_amdgcn_perm(vw[1], vw[0], 0x07060302u);
      const uint32_t vhi1 = __builtin_amdgcn_perm(vw[3], vw[2], 0x07060302u);
      const int v2 = 2 * (tid & 31), t4 = 4 * (tid >> 5);
      *reinterpret_cast<uint2*>(sVT + v2 * SV + ilv(t4)) = make_uint2(vlo0, vlo1);
      *reinterpret_cast<uint2*>(sVT + (v2 + 1) * SV + ilv(t4)) = make_uint2(vhi0, vhi1);
    }
    if (w == 0) {
      const float x = chunk_log2_decay(graw, lane);
      const float gc = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), C - 1));
      if (lane < C) {
        bEG(b)[lane] = ex2(x);
        bEH(b)[lane] = ex2(gc - x);
      }
    }
  };
  // -T' of a chunk, straight into the U phase's A operands (hi, lo per row tile)
  uint4 tpr[4];
  auto fetch_tp = [&](int ci) {
#pragma unroll
    for (int e = 0; e < 4; ++e) tpr[e] = tp[int64_t(ci) * TP_VEC + e * 64 + lane];
  };

  // S' split into bf16 hi + lo in the B-operand order of X's four contraction steps: formed
  // right after each update, where it overlaps the update's last MFMAs, so that X of the
  // next chunk starts on its products as soon as the chunk is staged
  bf16x8 s_hi[4], s_lo[4];
  auto split_state = [&]() {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      float x[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = S[2 * kk + (e >> 2)][e & 3];
      split8(x, s_hi[kk], s_lo[kk]);
    }
  };

  // prologue: chunk 0 staged, chunk 1 and the first factors in flight
  fetch(0);
  stage(0);
  fetch(C);
  fetch_tp(0);
  split_state();
  __syncthreads();

  for (int t0 = 0, b = 0, ci = 0; t0 < W; t0 += C, b ^= 1, ++ci) {
    // ---- X = Diag(2^G) (K S') on this wave's columns ---------------------------------
    f32x4 X[2] = {};
    {
      const __bf16* sK = reinterpret_cast<const __bf16*>(bK(b));
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
#pragma unroll
        for (int mu = 0; mu < 2; ++mu) {
          const bf16x8 kk8 = ld16(sK + (16 * mu + r) * SK + 32 * kk + 8 * q);
          X[mu] = mma(kk8, s_lo[kk], X[mu]);
          X[mu] = mma(kk8, s_hi[kk], X[mu]);
        }
      }
#pragma unroll
      for (int mu = 0; mu < 2; ++mu) X[mu] *= *reinterpret_cast<const f32x4*>(bEG(b) + 16 * mu + 4 * q);
    }

    // ---- U = (-T')(X - V), Diag(2^{G_C - G}) U, S' <- 2^{G_C} S' + K^T U ----------------
    {
      const uint16_t* sVT = bVT(b);
      const float* sEH = bEH(b);
      f32x4 U[2];
      bf16x8 yh, yl;
      float x[8];
      // this lane's column at tokens 4q .. 4q + 3 (mu = 0) and 16 + 4q .. (mu = 1)
      const uint4 v4 = *reinterpret_cast<const uint4*>(sVT + (16 * w + r) * SV + 8 * q);
      const uint32_t vw4[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
      for (int mu = 0; mu < 2; ++mu) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          x[4 * mu + i] = dot2(as_bf2(vw4[2 * mu + (i >> 1)]), (i & 1) ? kNegHi : kNegLo, X[mu][i]);
      }
      split8(x, yh, yl);
#pragma unroll
      for (int mu = 0; mu < 2; ++mu) {
        const bf16x8 ah = __builtin_bit_cast(bf16x8, tpr[2 * mu]);
        const bf16x8 al = __builtin_bit_cast(bf16x8, tpr[2 * mu + 1]);
        f32x4 c = mma(al, yh, f32x4{0.f, 0.f, 0.f, 0.f});
        c = mma(ah, yl, c);
        U[mu] = mma(ah, yh, c);
        U[mu] *= *reinterpret_cast<const f32x4*>(sEH + 16 * mu + 4 * q);
      }
      if (t0 + C < W) fetch_tp(ci + 1);
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
        const bf16x8 kt8 = ld16(sKT + (16 * mt + r) * SV + 8 * q);
        S[mt] = mma(kt8, ul, S[mt] * gam);
        S[mt] = mma(kt8, uh, S[mt]);
      }
      split_state();   // (after the last chunk: unused)
    }

    // ---- the next chunk into the other buffer; the one after that into registers --------
    if (t0 + C < W) {
      stage(b ^ 1);
      if (t0 + 2 * C < W) fetch(t0 + 2 * C);
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

inline int gdn_chunks(int W) { return (W + C - 1) / C; }

void launch_factors(int n_req, int H, int Hqk, int layer, const int32_t* inv_row, const uint16_t* k,
                    const float* g, const float* beta, int W, void* ws, hipStream_t st) {
  const int n_chunks = gdn_chunks(W);
  const dim3 grid(unsigned(n_req) * unsigned(H) * unsigned((n_chunks + 3) / 4)), block(256);
  hipLaunchKernelGGL(gdn_factor_kernel, grid, block, 0, st, H, Hqk, layer, inv_row, k, g, beta, W,
                     n_chunks, static_cast<uint4*>(ws));
}

}  // namespace

namespace dasc {

size_t gdn_factor_workspace_bytes(int n_req, int H, int W) {
  return size_t(n_req) * size_t(H) * size_t(gdn_chunks(W)) * size_t(kGdnFactorBytesPerChunk);
}

int64_t gdn_factor_blocks(int n_req, int H, int W) {
  return int64_t(n_req) * H * ((gdn_chunks(W) + 3) / 4);
}

void launch_refresh_wy_gdn(int n_req, int H, int Hqk, int layer, int L, const int32_t* inv_row,
                           float* states, int64_t n_pool, const int32_t* slot, const uint16_t* k,
                           const uint16_t* v, const float* g, const float* beta, int W,
                           int init_zero, void* ws, hipStream_t st) {
  launch_factors(n_req, H, Hqk, layer, inv_row, k, g, beta, W, ws, st);
  const dim3 grid(unsigned(n_req) * unsigned(H) * 2u), block(256);
  const CkptView none{nullptr, 1, 1, 0, nullptr};
  hipLaunchKernelGGL(refresh_wy_gdn_kernel<false>, grid, block, 0, st, H, Hqk, layer, L, inv_row,
                     states, n_pool, slot, k, v, g, W, init_zero, none,
                     static_cast<const uint4*>(ws), gdn_chunks(W));
}

void launch_restore_refresh_wy_gdn(int n_req, int H, int Hqk, int layer, int L, const float* ckpt,
                                   int64_t n_ckpt_slots, const int32_t* ck_slot,
                                   int64_t slice_rows, int64_t n_rows, const int32_t* inv_row,
                                   float* states, int64_t n_pool, const int32_t* slot,
                                   const uint16_t* k, const uint16_t* v, const float* g,
                                   const float* beta, int W, int init_zero, void* ws,
                                   hipStream_t st) {
  launch_factors(n_req, H, Hqk, layer, inv_row, k, g, beta, W, ws, st);
  const dim3 grid(unsigned(n_req) * unsigned(H) * 2u), block(256);
  const CkptView ck{ckpt, n_ckpt_slots, slice_rows, n_rows, ck_slot};
  hipLaunchKernelGGL(refresh_wy_gdn_kernel<true>, grid, block, 0, st, H, Hqk, layer, L, inv_row,
                     states, n_pool, slot, k, v, g, W, init_zero, ck,
                     static_cast<const uint4*>(ws), gdn_chunks(W));
}

}  // namespace dasc
