// Chunkwise WY-form refresh kernel on bf16 MFMA (gfx950), dk = dv = 128.
//
// Same recurrence as the per-column kernel (Sec. 3.1, Eq. 1 on S' = S^T):
//     S~ = Diag(exp(g_t)) S'_{t-1},   S'_t = S~ + beta_t k_t (v_t - S~^T k_t)^T.
// Unrolled over a chunk of C = 32 tokens with G_t = sum_{r<=t} g_r (per channel):
//     A_ts = beta_t sum_c k_tc k_sc exp(G_tc - G_sc)      (s < t)
//     T    = (I + A)^{-1},   T' = T Diag(beta)
//     U    = T' (V - K_G S')          K_G = k * exp(G)         (per-token deltas)
//     S'  <- Diag(exp(G_C)) S' + K_H^T U   K_H = k * exp(G_C - G)
// which is the per-token rule exactly, up to rounding.
//
// Work split: one 256-thread block per (request, head); wave w owns value columns
// [32w, 32w + 32) of S' (128 x 32 fp32 = 16 MFMA accumulator tiles held in VGPRs for
// the whole replay), tile nt holding the columns 32w + 2r + nt (r = lane % 16), so that
// a lane's values for both tiles are one 32-bit word per token.  Everything that does not
// depend on S' (cumulative decays, K_G, K_H, A, T') is built cooperatively in LDS each
// chunk; then each wave runs its three chained contractions K_G S', T'(V - .), K_H^T U on
// its own columns.  The chunk's decays, K_G, Q and K_H are formed at the end of the
// previous chunk, between its update products (K_G and Q go to LDS at once, K_H^T waits in
// registers until every wave is done with the previous one), so that a chunk starts with A
// and takes two barriers.
//
// Precision.  The products run on bf16 MFMA (16x16x32; 16x16x16 for the diagonal blocks
// of T) with fp32 accumulation.  An fp32 operand x is split into x_hi = bf16(x) and
// x_lo = bf16(x - x_hi); a product is formed as a_lo b_hi + a_hi b_lo + a_hi b_hi, which
// keeps ~16 mantissa bits per term.  This is what lets an fp32 state survive thousands
// of tokens within 2e-3 while running at the bf16 matrix-core rate.
//
// Register-resident chaining.  In the 16x16x32 layout lane (q = lane/16, r = lane%16)
// holds A[m = r][k = 8q + e], B[k = 8q + e][n = r] and D[m = 4q + i][n = r].  The
// contraction index can be any bijection shared by A and B, so an accumulator pair of
// 16-row tiles is fed straight back as a B operand by taking k(q, e) = 4q + e (e < 4)
// and 16 + 4q + (e - 4) (e >= 4); the LDS-side operand is read with the same mapping.
// S', K_G S', V - K_G S' and U never leave registers.
//
// LDS rows are padded so that the 16 (or 32) rows touched by one access instruction
// fall on distinct banks; every operand is read as a 16- or 8-byte vector.
//
// Decay factors.  exp(G_t - G_s) <= 1 for s <= t, but a factorised form needs
// exp(G_t - G_ref) exp(G_ref - G_s).  Fast path: when every channel decays by at most
// 2^96 over the chunk (a block-wide test per chunk; realistic gates decay far less),
// the reference is the chunk start: A = Diag(beta) strictly-lower(K_G Q^T) with
// K_G = k 2^G (which X needs anyway) and Q = k 2^{-G} <= 2^96 |k|, so the chunk takes
// two exponentials per (token, channel) for A and one for K_H, all formed by the thread
// that holds the gates in registers.  Strong-decay path otherwise: off-diagonal 16-token
// blocks use the block boundary as reference (both factors <= 1); diagonal blocks use the
// block midpoint, whose factors are bounded by exp(8 |g|max).  Per-token log-gates are
// floored at -10 (a decay of 4.5e-5 per token instead of anything smaller), which keeps
// every factor below e^80 in fp32 and changes the state by at most 4.5e-5 of its
// magnitude per floored token.
//
// Fused with the restore (FUSED = true), the initial state of a head is read from the
// packed checkpoint instead of the active state (kept rows from their packed position,
// omitted rows +0.0), and every row of the layer is written: kept rows first, copied bit
// for bit from the checkpoint in one 16-byte-per-thread pass whose stores drain while the
// replay runs, omitted rows from the replay at the end.  A head with no omitted row is a
// plain copy.  The arithmetic is the unfused kernel's, so the result equals restore
// followed by refresh bit for bit.  (Storing the kept rows from the registers that load
// the initial state instead keeps those values live into the replay and makes it spill.)
//
// Inputs are read through raw buffer resources sized to one head's window, so tokens
// past the window load as zeros: k = v = 0, g = 0, beta = 0, an identity step.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "ckpt_layout.h"
#include "refresh_kernels.h"
#include "wy_ops.h"

namespace {

using namespace dasc_wy;

constexpr int C = 32;       // tokens per chunk
constexpr int D = 128;      // dk = dv
constexpr float kGateFloor = -10.f;
// Fast path bound: every channel's log2-decay over a chunk at least -kFastRange, so that
// k 2^G and k 2^{-G} stay normal fp32 (and their bf16 low parts too) for every token.
constexpr float kFastRange = 96.f;
constexpr float kLog2e = 1.4426950408889634f;

// padded row strides (elements)
constexpr int SG = 132;     // f32 [C][SG]   cumulative log2-decay
constexpr int SK = 136;     // bf16 [C][SK]  keys, K_G
constexpr int SV = 40;      // bf16 [D][SV]  K_H^T
constexpr int SP = 36;      // bf16 [C][SP]  diagonal blocks of T' (8-byte aligned rows)
constexpr int ST = 36;      // f32  [C][ST]  A, then the diagonal blocks of T

// LDS map (bytes).  The key buffer is dead once A and K_H are built and then holds the
// diagonal blocks of T'.  On the fast path the gate buffer holds Q (hi, lo) instead.
// The A buffer keeps block (1, 0) of A; each diagonal block of A is replaced by the same
// block of T.
constexpr int G_BYTES = C * SG * 4 > 2 * C * SK * 2 ? C * SG * 4 : 2 * C * SK * 2;
constexpr int OFF_G = 0;                       // f32  [C][SG]; fast path: bf16 [2][C][SK] Q (ilv)
constexpr int OFF_K = OFF_G + G_BYTES;         // bf16 [C][SK]  -> later T' diagonal blocks
constexpr int OFF_TPH = OFF_K;                 // bf16 [C][SP]
constexpr int OFF_TPL = OFF_TPH + C * SP * 2;
constexpr int OFF_KGH = OFF_K + C * SK * 2;    // bf16 [C][SK], channels interleaved (ilv)
constexpr int OFF_KGL = OFF_KGH + C * SK * 2;
constexpr int OFF_KHH = OFF_KGL + C * SK * 2;  // bf16 [D][SV], tokens interleaved (ilv)
constexpr int OFF_KHL = OFF_KHH + D * SV * 2;
constexpr int OFF_A = OFF_KHL + D * SV * 2;    // f32  [C][ST]
// Per-chunk scalars alternate between two copies by chunk parity, so that a chunk can
// stage them while the waves still finishing the previous one read theirs.
constexpr int OFF_BETA = OFF_A + C * ST * 4;   // f32  [2][C]
constexpr int OFF_GAM = OFF_BETA + 2 * C * 4;  // f32  [2][D] exp(G_C)
constexpr int OFF_FLAGS = OFF_GAM + 2 * D * 4; // int  [2][4] per wave: fast path possible
constexpr int OFF_OMIT = OFF_FLAGS + 2 * 4 * 4;  // u8 [D] row omitted (replayed)
constexpr int LDS_BYTES = OFF_OMIT + D;
static_assert(2 * C * SP * 2 <= C * SK * 2, "T' must fit in the key buffer");
static_assert(LDS_BYTES <= 81920, "two blocks per CU");

__device__ inline float bf2f(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// Packed checkpoint of the fused variant (unused when FUSED is false).
using dasc::CkptView;

template <bool PER_CHANNEL, bool FUSED>
__global__ __launch_bounds__(256, 2) void refresh_wy_kernel(
    int H, int Hqk, int layer, int L, const int32_t* __restrict__ inv_row,
    float* __restrict__ states, int64_t n_pool, const int32_t* __restrict__ slot,
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ v, const float* __restrict__ g,
    const float* __restrict__ beta, int W, int init_zero, CkptView ck) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[LDS_BYTES];
  float* sG = reinterpret_cast<float*>(smem + OFF_G);
  uint16_t* sK = reinterpret_cast<uint16_t*>(smem + OFF_K);
  __bf16* sKGH = reinterpret_cast<__bf16*>(smem + OFF_KGH);
  __bf16* sKGL = reinterpret_cast<__bf16*>(smem + OFF_KGL);
  __bf16* sKHH = reinterpret_cast<__bf16*>(smem + OFF_KHH);
  __bf16* sKHL = reinterpret_cast<__bf16*>(smem + OFF_KHL);
  float* sA = reinterpret_cast<float*>(smem + OFF_A);
  __bf16* sTPH = reinterpret_cast<__bf16*>(smem + OFF_TPH);
  __bf16* sTPL = reinterpret_cast<__bf16*>(smem + OFF_TPL);
  float* const sBeta2 = reinterpret_cast<float*>(smem + OFF_BETA);
  float* const sGam2 = reinterpret_cast<float*>(smem + OFF_GAM);
  int* const sFast2 = reinterpret_cast<int*>(smem + OFF_FLAGS);
  unsigned char* const sOmit = smem + OFF_OMIT;
  __bf16* sQH = reinterpret_cast<__bf16*>(smem + OFF_G);   // fast path only
  __bf16* sQL = sQH + C * SK;

  const int n = blockIdx.x / H;
  const int h = blockIdx.x - n * H;
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int q = lane >> 4, r = lane & 15;

  const int64_t head_row = (int64_t(layer) * H + h) * D;
  bool mine = false;
  if (tid < D) {
    mine = inv_row[head_row + tid] < 0;
    sOmit[tid] = mine;
  }
  const bool any_omitted = __syncthreads_or(mine);
  if (!FUSED && !any_omitted) return;
  const int64_t sl = slot[n];
  if (sl < 0 || sl >= n_pool) return;
  float* S_head = states + (sl * L * H * D + head_row) * D;
  int64_t cslot = 0;
  if (FUSED) {
    cslot = ck.slot[n];
    if (cslot < 0 || cslot >= ck.n_slots) return;
  }
  // Fused: where dense row c of this head sits in the checkpoint, as a float offset
  // (kOmitted for an omitted row, kNoRow for an index outside the packed rows, which
  // restores as +0.0).  One thread per row fills the table in the A buffer, which is
  // free until the first chunk.
  using dasc::kOmitted;
  int64_t* sOff = reinterpret_cast<int64_t*>(smem + OFF_A);
  static_assert(D * 8 <= C * ST * 4, "row table must fit in the A buffer");
  if (FUSED) {
    if (tid < D) sOff[tid] = dasc::ckpt_row_offset(inv_row[head_row + tid], ck, cslot, D);
    __syncthreads();
  }
  if (FUSED) {
    // Every row that is not replayed is final already: its checkpoint row (or +0.0) is
    // copied to the pool here, 16 bytes per thread and access, and the stores drain
    // while the replay runs.  A head with no omitted row is done after this.
    for (int e = tid; e < D * D / 4; e += 256) {
      const int c = e >> 5, v4 = e & 31;
      const int64_t o = sOff[c];
      if (!any_omitted || o != kOmitted) {
        const f32x4 val = o >= 0 ? reinterpret_cast<const f32x4*>(ck.ckpt + o)[v4]
                                 : f32x4{0.f, 0.f, 0.f, 0.f};
        reinterpret_cast<f32x4*>(S_head + int64_t(c) * D)[v4] = val;
      }
    }
    if (!any_omitted) return;
  }

  // S'[c][j] for c = 16 mt + 4q + i, j = 32w + 2r + nt: the lane's two columns of a row
  // are adjacent, one 8-byte load
  f32x4 S[8][2];
#pragma unroll
  for (int mt = 0; mt < 8; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = 16 * mt + 4 * q + i, j = 32 * w + 2 * r;
      f32x2 val = {0.f, 0.f};
      if (FUSED) {
        const int64_t o = sOff[c];   // the restored value: kept row, or +0.0
        if (!init_zero && o >= 0) val = *reinterpret_cast<const f32x2*>(ck.ckpt + o + j);
      } else if (!init_zero) {
        val = *reinterpret_cast<const f32x2*>(S_head + int64_t(c) * D + j);
      }
      S[mt][0][i] = val[0];
      S[mt][1][i] = val[1];
    }

  const int hk = h / (H / Hqk);
  const uint16_t* kp = k + (int64_t(n) * Hqk + hk) * W * D;
  const uint16_t* vp = v + (int64_t(n) * H + h) * W * D;
  const float* gp = PER_CHANNEL ? g + (int64_t(n) * H + h) * W * D : g + (int64_t(n) * H + h) * W;
  const float* bp = beta + (int64_t(n) * H + h) * W;
  const __amdgpu_buffer_rsrc_t rk = rsrc(kp, W * D * 2), rv = rsrc(vp, W * D * 2);
  const __amdgpu_buffer_rsrc_t rg = rsrc(gp, PER_CHANNEL ? W * D * 4 : W * 4), rb = rsrc(bp, W * 4);

  // Load phase: thread (cq = tid / 8, og = tid % 8) owns channels 4 cq .. 4 cq + 3 at the
  // four tokens 4 og .. 4 og + 3 of a chunk.  It loads their gates and keys one chunk
  // ahead and forms the running sums of the gates (the eight token groups of a channel
  // quad are eight adjacent lanes); on the fast path it also builds their entries of K_G,
  // Q and K_H from its registers, each written as one 8-byte store per token or channel
  // (a wave's stores then fall on distinct LDS banks).
  const int cq = tid >> 3, og = tid & 7;
  const int c4 = 4 * cq, t4 = 4 * og;

  // Gates, keys and beta of one chunk as this thread loads them; the next chunk's are
  // issued one chunk ahead.
  f32x4 graw[4];
  uint2 kq[4];
  float braw;
  auto fetch_g = [&](int c0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (PER_CHANNEL) {
        graw[i] = ldf4(rg, ((t4 + i) * D + c4) * 4, c0 * D * 4);
      } else {
        const float x = ldf(rg, (t4 + i) * 4, c0 * 4);
        graw[i] = f32x4{x, x, x, x};
      }
    }
    braw = ldf(rb, (tid & (C - 1)) * 4, c0 * 4);
  };
  auto fetch_k = [&](int c0) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      kq[i] = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(
                                            rk, ((t4 + i) * D + c4) * 2, c0 * D * 2, 0));
  };
  // Values stay in registers in the layout the U phase consumes: lane (q, r) of wave w
  // holds, for tokens 16 mu + 4q + i, the word with columns 32w + 2r (low half) and
  // 32w + 2r + 1 (high half) -- its two S' tiles.  The next chunk's are loaded as soon as
  // U has read this chunk's.
  uint32_t vreg[2][4];
  auto fetch_v = [&](int c0) {
#pragma unroll
    for (int mu = 0; mu < 2; ++mu)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        vreg[mu][i] = __builtin_amdgcn_raw_buffer_load_b32(
            rv, ((16 * mu + 4 * q + i) * D + 32 * w + 2 * r) * 2, c0 * D * 2, 0);
  };
  // X = K_G S' on this wave's columns (rows t, contraction over channels), one step per
  // 32 channels
  f32x4 X[2][2];
  auto x_step = [&](int kk) {
    bf16x8 sh[2], slo[2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      float x[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = S[2 * kk + (e >> 2)][nt][e & 3];
      split8(x, sh[nt], slo[nt]);
    }
#pragma unroll
    for (int mu = 0; mu < 2; ++mu) {
      const int o = (16 * mu + r) * SK + 32 * kk + 8 * q;
      const bf16x8 ah = ld16(sKGH + o), al = ld16(sKGL + o);
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) X[mu][nt] = mma3(ah, al, sh[nt], slo[nt], X[mu][nt]);
    }
  };
  auto x_init = [&]() {
#pragma unroll
    for (int mu = 0; mu < 2; ++mu)
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) X[mu][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  };
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};
  // left * right for 16x16 blocks in the accumulator layout (lane (q, r) holds rows 4q + i
  // of column r), on bf16 MFMA (16x16x16): each block split hi/lo into two packed words,
  // which is exactly that MFMA's operand layout for the left factor's transpose and for
  // the right factor, so products chain without leaving registers; three products
  // l_lo r_hi + l_hi r_lo + l_hi r_hi, as for every other product here.
  struct Split4 { uint2 h, l; };
  auto split4 = [](const f32x4 x) {
    Split4 s;
    split2(x[0], x[1], s.h.x, s.l.x);
    split2(x[2], x[3], s.h.y, s.l.y);
    return s;
  };
  auto mulb = [](const Split4& lt, const Split4& rt, f32x4 c) {
    c = mma16(lt.l, rt.h, c);
    c = mma16(lt.h, rt.l, c);
    return mma16(lt.h, rt.h, c);
  };
  // Running sums of one chunk's gates (log2 units, floored) at this thread's four tokens
  // and channels, and the chunk totals.  Lanes 8 cq .. 8 cq + 7 hold the eight token groups
  // of a channel quad: within a lane quad, the values shifted up by one lane (zero into the
  // first) are summed by two shift-and-add steps; the upper quad adds the lower quad's
  // total (row shift of 4); all eight lanes form the chunk total as (lower total) + (upper
  // total).  The selects are bitwise (all-ones / zero lane masks): a conditional expression
  // lets the compiler move a DPP read under an exec mask, where a lane whose source lane is
  // masked off reads a stale value.
  auto gate_sums = [&](const f32x4 (&gr)[4], f32x4 (&Gl)[4], f32x4& gc) {
    f32x4 run = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int j = 0; j < 4; ++j) run[j] += fmaxf(gr[i][j], kGateFloor) * kLog2e;
      Gl[i] = run;
    }
    const uint32_t m_first = (og & 3) == 0 ? ~0u : 0u, m_upper = og >= 4 ? ~0u : 0u;
    f32x4 x, base;
#pragma unroll
    for (int j = 0; j < 4; ++j) x[j] = bsel(m_first, 0.f, quad_perm<0x90>(run[j]));   // [0,0,1,2]
#pragma unroll
    for (int j = 0; j < 4; ++j) x[j] += quad_perm<0x90>(x[j]);
#pragma unroll
    for (int j = 0; j < 4; ++j) x[j] += quad_perm<0x40>(x[j]);                        // [0,0,0,1]
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float tq = quad_perm<0xFF>(x[j] + run[j]);                                 // [3,3,3,3]
      const float below = row_shr<4>(tq), above = row_shl<4>(tq);
      base[j] = x[j] + bsel(m_upper, below, 0.f);
      gc[j] = bsel(m_upper, below + tq, tq + above);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) Gl[i] += base;
  };

  // K_H^T of the next chunk (rows c4 + j, tokens t4 .. t4 + 3, hi and lo), held in
  // registers until every wave is done with this chunk's.
  uint2 khh[4], khl[4];
  // Everything of a chunk that does not depend on S', staged at the end of the previous
  // chunk (its gates and keys are in registers by then): beta, 2^{G_C} and the per-wave
  // fast-path flags into the chunk's parity copies, and the fast-path factors K_G = k 2^G
  // and Q = k 2^{-G} into their buffers (free once every wave has formed the previous
  // chunk's A and X).  When the chunk takes the strong-decay path instead, that path
  // rebuilds every factor and these values are overwritten unused.
  auto prepare = [&](int par) {
    float* const sBeta = sBeta2 + par * C;
    float* const sGam = sGam2 + par * D;
    int* const sFast = sFast2 + par * 4;
    f32x4 Gl[4], gc;
    gate_sums(graw, Gl, gc);
    if (tid < C) sBeta[tid] = braw;
    f32x4 gam;   // 2^{G_C} on channels c4 .. c4 + 3
#pragma unroll
    for (int j = 0; j < 4; ++j) gam[j] = ex2(gc[j]);
    if (og == 7) *reinterpret_cast<f32x4*>(sGam + c4) = gam;
    {
      const float gmin = fminf(fminf(gc[0], gc[1]), fminf(gc[2], gc[3]));
      const int wave_fast = __all(gmin >= -kFastRange);
      if (lane == 0) sFast[w] = wave_fast;
    }
    float kf[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      kf[i][0] = __uint_as_float(kq[i].x << 16);
      kf[i][1] = __uint_as_float(kq[i].x & 0xFFFF0000u);
      kf[i][2] = __uint_as_float(kq[i].y << 16);
      kf[i][3] = __uint_as_float(kq[i].y & 0xFFFF0000u);
    }
    float qf[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int o = (t4 + i) * SK + ilv(c4);
      float kg[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        kg[j] = kf[i][j] * ex2(Gl[i][j]);
        qf[i][j] = kf[i][j] * ex2(-Gl[i][j]);
      }
      uint2 hi, lo;
      split2(kg[0], kg[1], hi.x, lo.x);
      split2(kg[2], kg[3], hi.y, lo.y);
      *reinterpret_cast<uint2*>(sKGH + o) = hi;
      *reinterpret_cast<uint2*>(sKGL + o) = lo;
      split2(qf[i][0], qf[i][1], hi.x, lo.x);
      split2(qf[i][2], qf[i][3], hi.y, lo.y);
      *reinterpret_cast<uint2*>(sQH + o) = hi;
      *reinterpret_cast<uint2*>(sQL + o) = lo;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {   // K_H^T = (Q 2^{G_C})^T
      split2(qf[0][j] * gam[j], qf[1][j] * gam[j], khh[j].x, khl[j].x);
      split2(qf[2][j] * gam[j], qf[3][j] * gam[j], khh[j].y, khl[j].y);
    }
  };

  // Issued in the order the loop issues them (keys, gates, values), so that each wait
  // counts only older loads.
  __builtin_amdgcn_sched_barrier(0);
  fetch_k(0);
  __builtin_amdgcn_sched_barrier(0);
  fetch_g(0);
  __builtin_amdgcn_sched_barrier(0);
  fetch_v(0);
  __builtin_amdgcn_sched_barrier(0);
  prepare(0);
  fetch_k(C);
  fetch_g(C);

  // Two blocks share a CU, and the instruction arbiter prefers the older block's waves: left
  // alone, the block placed first runs its chunks ~1.5x as fast as the other, which then
  // finishes alone.  The later half of the grid (placed second) takes the higher wave
  // priority for its first 60% of chunks, the earlier half for the rest, so that the pair
  // finishes at about the same time.
  const int second = __builtin_amdgcn_readfirstlane(blockIdx.x >= (gridDim.x + 1) / 2 ? 1 : 0);
  const int t_flip = ((W + C - 1) / C * 3 / 5) * C;
  for (int t0 = 0; t0 < W; t0 += C) {
    if ((t0 < t_flip) == (second != 0)) __builtin_amdgcn_s_setprio(1);
    else __builtin_amdgcn_s_setprio(0);
    const int par = (t0 / C) & 1;
    float* const sBeta = sBeta2 + par * C;
    float* const sGam = sGam2 + par * D;
    int* const sFast = sFast2 + par * 4;
    // this chunk's staged scalars and fast-path factors are complete, and every wave is done
    // with the previous chunk
    __syncthreads();
    const int4 fl = *reinterpret_cast<const int4*>(sFast);
    const bool fast = fl.x && fl.y && fl.z && fl.w;

    // Waves 0 and 2 hold diagonal block w / 2 of A and its transpose in the accumulator
    // layout (a, at); wave 1 leaves block (1, 0) of A in the A buffer.
    f32x4 a = zero4, at = zero4;
    if (fast) {
      // ---- fast path: K_H^T from the registers (read only after the next barrier); K_G and
      // Q are in LDS already
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        *reinterpret_cast<uint2*>(sKHH + (c4 + j) * SV + ilv(t4)) = khh[j];
        *reinterpret_cast<uint2*>(sKHL + (c4 + j) * SV + ilv(t4)) = khl[j];
      }

      // ---- A = Diag(beta) (strictly lower part of K_G Q^T): waves 0 and 2 a diagonal block,
      // and its transpose by a round trip through their own corner of the A buffer (the
      // wave reads back what it wrote, so no block barrier); wave 1 block (1, 0).
      if (w < 3) {
        const int ti = w == 0 ? 0 : 1, si = w == 2 ? 1 : 0;
        const int tr = 16 * ti + r, sr = 16 * si + r;
        const f32x4 bt = *reinterpret_cast<const f32x4*>(sBeta + 16 * ti + 4 * q);
        f32x4 acc = zero4, acc2 = zero4;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const int ot = tr * SK + 32 * kk + 8 * q, os = sr * SK + 32 * kk + 8 * q;
          const bf16x8 ah = ld16(sKGH + ot), al = ld16(sKGL + ot);
          const bf16x8 bh = ld16(sQH + os), bl = ld16(sQL + os);
          if (kk & 1) acc2 = mma3(ah, al, bh, bl, acc2);
          else acc = mma3(ah, al, bh, bl, acc);
        }
        acc += acc2;
        if (w == 1) {
#pragma unroll
          for (int i = 0; i < 4; ++i) sA[(16 + 4 * q + i) * ST + r] = bt[i] * acc[i];
        } else {
          const int base = 8 * w;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            a[i] = r < 4 * q + i ? bt[i] * acc[i] : 0.f;    // A[base + 4q + i][base + r]
            sA[(base + 4 * q + i) * ST + base + r] = a[i];
          }
          wave_lds_sync();
#pragma unroll
          for (int i = 0; i < 4; ++i) at[i] = sA[(base + r) * ST + base + 4 * q + i];   // A[base + r][base + 4q + i]
        }
      }
    } else {
      // ---- strong-decay path ------------------------------------------------------------
      // this chunk's gates and keys again (the registers hold the next chunk's by now), and
      // their running decays, into LDS row-major
      {
        f32x4 gr[4], Gl[4], gc;
        uint2 kc[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (PER_CHANNEL) {
            gr[i] = ldf4(rg, ((t4 + i) * D + c4) * 4, t0 * D * 4);
          } else {
            const float x = ldf(rg, (t4 + i) * 4, t0 * 4);
            gr[i] = f32x4{x, x, x, x};
          }
          kc[i] = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(
                                                rk, ((t4 + i) * D + c4) * 2, t0 * D * 2, 0));
        }
        gate_sums(gr, Gl, gc);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          *reinterpret_cast<f32x4*>(sG + (t4 + i) * SG + c4) = Gl[i];
          *reinterpret_cast<uint2*>(sK + (t4 + i) * SK + c4) = kc[i];
        }
      }
      __syncthreads();
      // A = Diag(beta) (strictly lower part of R Q^T), three 16x16 tiles on bf16 MFMA
      // (16x16x32) with hi/lo split factors, like the state products: lane (q, r) feeds
      // channels 32 kk + 8 q + e of its row to step kk (three MFMAs a step where fp32 MFMA
      // would take eight, at a sixteenth of the bf16 rate).  Each tile factors the decay
      // at its own reference token, so no factor exceeds 2^{8 |g|max}.
      if (w < 3) {
        const int ti = w == 0 ? 0 : 1, si = w == 2 ? 1 : 0;
        const int rf = w == 0 ? 8 : (w == 1 ? 15 : 24);   // reference token of the tile
        const int tr = 16 * ti + r, sr = 16 * si + r;
        f32x4 acc = zero4, acc2 = zero4;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const int c0 = 32 * kk + 8 * q;
          float fa[8], fb[8];
#pragma unroll
          for (int h2 = 0; h2 < 2; ++h2) {
            const f32x4 gt = *reinterpret_cast<const f32x4*>(sG + tr * SG + c0 + 4 * h2);
            const f32x4 gs = *reinterpret_cast<const f32x4*>(sG + sr * SG + c0 + 4 * h2);
            const f32x4 gf = *reinterpret_cast<const f32x4*>(sG + rf * SG + c0 + 4 * h2);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              fa[4 * h2 + i] = ex2(gt[i] - gf[i]);
              fb[4 * h2 + i] = ex2(gf[i] - gs[i]);
            }
          }
          const uint4 kt = *reinterpret_cast<const uint4*>(sK + tr * SK + c0);
          const uint4 ks = *reinterpret_cast<const uint4*>(sK + sr * SK + c0);
          const uint32_t ktw[4] = {kt.x, kt.y, kt.z, kt.w}, ksw[4] = {ks.x, ks.y, ks.z, ks.w};
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            fa[e] *= __uint_as_float((e & 1) ? (ktw[e >> 1] & 0xFFFF0000u) : (ktw[e >> 1] << 16));
            fb[e] *= __uint_as_float((e & 1) ? (ksw[e >> 1] & 0xFFFF0000u) : (ksw[e >> 1] << 16));
          }
          bf16x8 ah, al, bh, bl;
          split8(fa, ah, al);
          split8(fb, bh, bl);
          if (kk & 1) acc2 = mma3(ah, al, bh, bl, acc2);
          else acc = mma3(ah, al, bh, bl, acc);
        }
        acc += acc2;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = 16 * ti + 4 * q + i;
          sA[t * ST + sr] = (ti == si && sr >= t) ? 0.f : sBeta[t] * acc[i];
        }
      } else {
        // meanwhile wave 3: K_H^T = (k exp(G_C - G))^T, rows = channels, split hi/lo
#pragma unroll
        for (int x = 0; x < 2; ++x) {
          const int c = lane + 64 * x;
          const float gC = sG[31 * SG + c];
#pragma unroll
          for (int m = 0; m < 4; ++m) {
            float x[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const int t = 8 * m + e;
              x[e] = bf2f(sK[t * SK + c]) * ex2(gC - sG[t * SG + c]);
            }
            bf16x8 hh, hl;
            split8(x, hh, hl);
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
              const int o = c * SV + ilv(8 * m + 4 * hf);
              *reinterpret_cast<bf16x4*>(sKHH + o) = bf16x4{hh[4 * hf], hh[4 * hf + 1], hh[4 * hf + 2], hh[4 * hf + 3]};
              *reinterpret_cast<bf16x4*>(sKHL + o) = bf16x4{hl[4 * hf], hl[4 * hf + 1], hl[4 * hf + 2], hl[4 * hf + 3]};
            }
          }
        }
      }
      // K_G = k exp(G), rows = tokens: two (token, 8-channel) units per thread (the keys
      // and gates are read here, before T' reuses the key buffer)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int t = (tid + 256 * u) >> 4, c8 = ((tid + 256 * u) & 15) * 8;
        const uint4 kr = *reinterpret_cast<const uint4*>(sK + t * SK + c8);
        const uint32_t kw[4] = {kr.x, kr.y, kr.z, kr.w};
        const f32x4 g0 = *reinterpret_cast<const f32x4*>(sG + t * SG + c8);
        const f32x4 g1 = *reinterpret_cast<const f32x4*>(sG + t * SG + c8 + 4);
        float x[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float kv = __uint_as_float((e & 1) ? (kw[e >> 1] & 0xFFFF0000u) : (kw[e >> 1] << 16));
          x[e] = kv * ex2(e < 4 ? g0[e & 3] : g1[e & 3]);
        }
        bf16x8 hh, hl;
        split8(x, hh, hl);
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const int o = t * SK + ilv(c8 + 4 * hf);
          *reinterpret_cast<bf16x4*>(sKGH + o) = bf16x4{hh[4 * hf], hh[4 * hf + 1], hh[4 * hf + 2], hh[4 * hf + 3]};
          *reinterpret_cast<bf16x4*>(sKGL + o) = bf16x4{hl[4 * hf], hl[4 * hf + 1], hl[4 * hf + 2], hl[4 * hf + 3]};
        }
      }
      __syncthreads();
      if (w == 0 || w == 2) {
        const int base = 8 * w;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          a[i] = sA[(base + 4 * q + i) * ST + base + r];
          at[i] = sA[(base + r) * ST + base + 4 * q + i];
        }
      }
    }

    // ---- diagonal blocks of T = (I + A)^{-1} on bf16 MFMA, and X = K_G S' ---------------
    // A strictly lower 16x16 block B has B^16 = 0, so (I + B)^{-1} = X1 X2 exactly with
    // X1 = (I - B)(I + B^2) and X2 = (I + B^4)(I + B^8): eight chained 16x16x16 products in
    // five dependent levels, each power carried together with its transpose.  A product
    // takes its factors split hi/lo on the 16x16x16 bf16 MFMA (three of them, the same three
    // terms as every other product here), a third of the matrix-pipe time of the four fp32
    // 16x16x4 MFMAs it replaces.  Waves 0 and 2 invert their block with the steps of X in
    // between (the two are independent, so the matrix pipe overlaps them); waves 1 and 3
    // only form X.
    x_init();
    if (w == 0 || w == 2) {
      const int base = 8 * w;
      f32x4 id;
#pragma unroll
      for (int i = 0; i < 4; ++i) id[i] = 4 * q + i == r ? 1.f : 0.f;
      const f32x4 imt = id - at;                           // (I - B)^T
      const Split4 sa = split4(a), sat = split4(at);
      const f32x4 p2 = mulb(sat, sa, zero4);               // B^2
      const f32x4 p2t = mulb(sa, sat, zero4);              // (B^2)^T
      x_step(0);
      const Split4 s2 = split4(p2), s2t = split4(p2t);
      const f32x4 p4 = mulb(s2t, s2, zero4);               // B^4
      const f32x4 p4t = mulb(s2, s2t, zero4);              // (B^4)^T
      const f32x4 x1t = mulb(s2, split4(imt), imt);        // X1^T = (I + B^2)^T (I - B)^T
      x_step(1);
      const Split4 s4t = split4(p4t);
      const f32x4 p8 = mulb(s4t, split4(p4), zero4) + id;  // I + B^8
      x_step(2);
      const f32x4 x2 = mulb(s4t, split4(p8), p8);          // X2
      x_step(3);
      const f32x4 tb = mulb(split4(x1t), split4(x2), zero4);   // T block: rows 4q + i, column r
      const float bs = sBeta[base + r];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = base + 4 * q + i;
        sA[t * ST + base + r] = tb[i];
        __bf16 hi, lo;
        split(-tb[i] * bs, hi, lo);   // -T' = -T Diag(beta)
        sTPH[t * SP + base + r] = hi;
        sTPL[t * SP + base + r] = lo;
      }
    } else {
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) x_step(kk);
    }
    __syncthreads();

    // ---- block (1, 0) of -T' = -T Diag(beta): T10 = -T11 A10 T00, formed by every wave as
    // its transpose T10^T = -T00^T (A10^T T11^T), which lands in the left-operand layout of
    // the U product (lane (q, r) register i: row r, token 4q + i).
    f32x4 tq;
    {
      f32x4 a10, t11t, t00;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a10[i] = sA[(16 + 4 * q + i) * ST + r];
        t11t[i] = sA[(16 + r) * ST + 16 + 4 * q + i];
        t00[i] = sA[(4 * q + i) * ST + r];
      }
      const f32x4 b4 = *reinterpret_cast<const f32x4*>(sBeta + 4 * q);
      tq = mulb(split4(t00), split4(mulb(split4(a10), split4(t11t), zero4)), zero4) * b4;
    }

    // ---- U = (-T')(X - V): the difference stays in registers as the B operand ------
    f32x4 U[2][2];
    {
      bf16x8 yh[2], yl[2];
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        float x[8];
#pragma unroll
        for (int mu = 0; mu < 2; ++mu)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            x[4 * mu + i] = dot2(as_bf2(vreg[mu][i]), nt ? kNegHi : kNegLo, X[mu][nt][i]);
          }
        split8(x, yh[nt], yl[nt]);
      }
      fetch_v(t0 + C);   // the next chunk's values (zeros past the window)
      uint2 qh, ql;
      split2(tq[0], tq[1], qh.x, ql.x);
      split2(tq[2], tq[3], qh.y, ql.y);
      const bf16x4 z4 = {};
      // rows 0..15: (T'00, 0); rows 16..31: (T'10, T'11)
      const int o0 = r * SP + 4 * q, o1 = (16 + r) * SP + 16 + 4 * q;
      const bf16x8 ah0 = cat(*reinterpret_cast<const bf16x4*>(sTPH + o0), z4);
      const bf16x8 al0 = cat(*reinterpret_cast<const bf16x4*>(sTPL + o0), z4);
      const bf16x8 ah1 = cat(__builtin_bit_cast(bf16x4, qh), *reinterpret_cast<const bf16x4*>(sTPH + o1));
      const bf16x8 al1 = cat(__builtin_bit_cast(bf16x4, ql), *reinterpret_cast<const bf16x4*>(sTPL + o1));
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        U[0][nt] = mma3(ah0, al0, yh[nt], yl[nt], zero4);
        U[1][nt] = mma3(ah1, al1, yh[nt], yl[nt], zero4);
      }
    }

    // ---- S' <- Diag(exp(G_C)) S' + K_H^T U ----------------------------------------------
    bf16x8 uh[2], ul[2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      float x[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = U[e >> 2][nt][e & 3];
      split8(x, uh[nt], ul[nt]);
    }
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) {
      const f32x4 gam = *reinterpret_cast<const f32x4*>(sGam + 16 * mt + 4 * q);
      const int o = (16 * mt + r) * SV + 8 * q;
      const bf16x8 ah = ld16(sKHH + o), al = ld16(sKHL + o);
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) S[mt][nt] = mma3(ah, al, uh[nt], ul[nt], S[mt][nt] * gam);
    }
    // ---- the next chunk's scalars and fast-path factors, between the update's products;
    // then the gates and keys of the chunk after it (zeros past the window)
    prepare(par ^ 1);
    fetch_k(t0 + 2 * C);
    fetch_g(t0 + 2 * C);
  }

#pragma unroll
  for (int mt = 0; mt < 8; ++mt) {
    // rows 16 mt + 4q .. 16 mt + 4q + 3: one omitted flag per byte
    const uint32_t om = *reinterpret_cast<const uint32_t*>(sOmit + 16 * mt + 4 * q);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = 16 * mt + 4 * q + i;
      if ((om >> (8 * i)) & 0xFFu) {
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) S_head[int64_t(c) * D + 32 * w + 2 * r + nt] = S[mt][nt][i];
      }
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
  const CkptView none{nullptr, 1, 1, 0, nullptr};
  if (per_channel)
    hipLaunchKernelGGL((refresh_wy_kernel<true, false>), grid, block, 0, st, H, Hqk, layer, L,
                       inv_row, states, n_pool, slot, k, v, g, beta, W, init_zero, none);
  else
    hipLaunchKernelGGL((refresh_wy_kernel<false, false>), grid, block, 0, st, H, Hqk, layer, L,
                       inv_row, states, n_pool, slot, k, v, g, beta, W, init_zero, none);
}

void launch_restore_refresh_wy(bool per_channel, int n_req, int H, int Hqk, int layer, int L,
                               const float* ckpt, int64_t n_ckpt_slots, const int32_t* ck_slot,
                               int64_t slice_rows, int64_t n_rows, const int32_t* inv_row,
                               float* states, int64_t n_pool, const int32_t* slot,
                               const uint16_t* k, const uint16_t* v, const float* g,
                               const float* beta, int W, int init_zero, hipStream_t st) {
  const dim3 grid(unsigned(n_req) * unsigned(H)), block(256);
  const CkptView ck{ckpt, n_ckpt_slots, slice_rows, n_rows, ck_slot};
  if (per_channel)
    hipLaunchKernelGGL((refresh_wy_kernel<true, true>), grid, block, 0, st, H, Hqk, layer, L,
                       inv_row, states, n_pool, slot, k, v, g, beta, W, init_zero, ck);
  else
    hipLaunchKernelGGL((refresh_wy_kernel<false, true>), grid, block, 0, st, H, Hqk, layer, L,
                       inv_row, states, n_pool, slot, k, v, g, beta, W, init_zero, ck);
}

}  // namespace dasc
