// Bounded-suffix refresh (DASC-WR, Sec. 4.2) of the gated delta-rule state (Eq. 1).
//
// The state of one head is stored transposed, S' = S^T in R^{dk x dv}; per token
//     S~   = Diag(exp(g_t)) S'_{t-1}
//     S'_t = S~ + beta_t k_t (v_t - S~^T k_t)^T
// Column j of S' (value channel j) evolves on its own: it needs k_t, g_t, beta_t and
// the single value v_t[j].  This kernel gives each thread one column, held in dk
// registers, so the dot product S~^T k_t is a private reduction and no lane ever
// waits on another.  A block owns one (request, head); k, the decays exp(g) and v
// for a tile of tokens are staged in LDS and read back as broadcasts.
//
// Per token and column this is dk multiplies (decay) and 2 dk FMAs (read-out and
// write), all fp32; it is bound by vector ALU throughput.  Only the omitted rows of
// the head (KDA) or the omitted heads (GDN) are written back; everything else in
// the active state keeps its bits.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "dasc.h"
#include "dasc_testing.h"
#include "launch_common.h"
#include "refresh_kernels.h"

namespace {

constexpr int kTile = 32;  // tokens staged per LDS tile

__device__ inline float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

template <int DK, bool PER_CHANNEL>
__global__ __launch_bounds__(256) void refresh_column_kernel(
    int H, int Hqk, int dv, int layer, int L, const int32_t* __restrict__ inv_row,
    float* __restrict__ states, int64_t n_pool, const int32_t* __restrict__ slot,
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ v, const float* __restrict__ g,
    const float* __restrict__ beta, int W, int init_zero) {
  __shared__ float k_s[kTile][DK];
  __shared__ float a_s[kTile][PER_CHANNEL ? DK : 1];
  __shared__ float b_s[kTile];
  extern __shared__ float v_s[];  // [kTile][dv]

  const int n = blockIdx.x / H;
  const int h = blockIdx.x - n * H;
  const int j = threadIdx.x;
  const int nthr = blockDim.x;

  const int64_t head_row = (int64_t(layer) * H + h) * DK;
  // Does this head have anything to refresh?
  bool mine = false;
  for (int c = j; c < DK; c += nthr) mine |= inv_row[head_row + c] < 0;
  if (!__syncthreads_or(mine)) return;
  const int64_t s = slot[n];
  if (s < 0 || s >= n_pool) return;

  float* S_head = states + (s * L * H * DK + head_row) * dv;
  const bool col = j < dv;
  float st[DK];
#pragma unroll
  for (int c = 0; c < DK; ++c) st[c] = (col && !init_zero) ? S_head[int64_t(c) * dv + j] : 0.f;

  const int hk = h / (H / Hqk);
  const uint16_t* kp = k + (int64_t(n) * Hqk + hk) * W * DK;
  const uint16_t* vp = v + (int64_t(n) * H + h) * W * dv;
  const float* gp = PER_CHANNEL ? g + (int64_t(n) * H + h) * W * DK : g + (int64_t(n) * H + h) * W;
  const float* bp = beta + (int64_t(n) * H + h) * W;

  for (int t0 = 0; t0 < W; t0 += kTile) {
    const int nt = min(kTile, W - t0);
    __syncthreads();
    for (int e = j; e < nt * DK; e += nthr) {
      const int tt = e / DK, c = e - tt * DK;
      k_s[tt][c] = bf16_to_f32(kp[int64_t(t0) * DK + e]);
      if (PER_CHANNEL) a_s[tt][c] = expf(gp[int64_t(t0) * DK + e]);
    }
    if (!PER_CHANNEL)
      for (int e = j; e < nt; e += nthr) a_s[e][0] = expf(gp[t0 + e]);
    for (int e = j; e < nt; e += nthr) b_s[e] = bp[t0 + e];
    for (int e = j; e < nt * dv; e += nthr) v_s[e] = bf16_to_f32(vp[int64_t(t0) * dv + e]);
    __syncthreads();

    for (int tt = 0; tt < nt; ++tt) {
      float y = 0.f;
#pragma unroll
      for (int c = 0; c < DK; ++c) {
        st[c] *= PER_CHANNEL ? a_s[tt][c] : a_s[tt][0];   // decay first
        y = fmaf(k_s[tt][c], st[c], y);                    // S~^T k_t
      }
      const float d = b_s[tt] * ((col ? v_s[tt * dv + j] : 0.f) - y);
#pragma unroll
      for (int c = 0; c < DK; ++c) st[c] = fmaf(k_s[tt][c], d, st[c]);  // + beta k (v - S~^T k)^T
    }
  }

  if (!col) return;
#pragma unroll
  for (int c = 0; c < DK; ++c)
    if (inv_row[head_row + c] < 0) S_head[int64_t(c) * dv + j] = st[c];
}

template <int DK>
void launch_column(bool per_channel, dim3 grid, dim3 block, size_t lds, hipStream_t st, int H,
                   int Hqk, int dv, int layer, int L, const int32_t* inv_row, float* states,
                   int64_t n_pool, const int32_t* slot, const uint16_t* k, const uint16_t* v,
                   const float* g, const float* beta, int W, int init_zero) {
  if (per_channel)
    hipLaunchKernelGGL((refresh_column_kernel<DK, true>), grid, block, lds, st, H, Hqk, dv, layer,
                       L, inv_row, states, n_pool, slot, k, v, g, beta, W, init_zero);
  else
    hipLaunchKernelGGL((refresh_column_kernel<DK, false>), grid, block, lds, st, H, Hqk, dv, layer,
                       L, inv_row, states, n_pool, slot, k, v, g, beta, W, init_zero);
}

// Does this shape take the two-launch scalar-gate GDN kernel?
bool uses_gdn_factors(const dasc_shape* shape) {
  return shape->arch == DASC_ARCH_GDN && dasc::refresh_wy_supported(shape->dk, shape->dv);
}

}  // namespace

extern "C" int dasc_refresh_workspace_bytes(const dasc_shape* shape, int32_t n_req, int32_t W,
                                            size_t* bytes) {
  if (!shape || !bytes || n_req < 1 || W < 1) return DASC_E_INVAL;
  if (!dasc::valid_shape(shape)) return DASC_E_SHAPE;
  // GDN heads at dk = dv = 128 keep each chunk's WY factor -T' between the two launches
  // of their kernel; every other path needs nothing.
  *bytes = uses_gdn_factors(shape)
               ? dasc::gdn_factor_workspace_bytes(n_req, shape->n_heads, W)
               : 0;
  return DASC_OK;
}

namespace dasc {

// dasc_refresh with an explicit kernel choice (DASC_REFRESH_KERNEL_*): AUTO takes the
// chunked MFMA kernels at dk = dv = 128 (the scalar-gate one for GDN heads) and the
// per-column fp32 kernel for every other shape.
int refresh_impl(const dasc_shape* shape, int32_t layer, const int32_t* inv_row, float* states,
                 int64_t n_pool, const int32_t* slot, const uint16_t* k, const uint16_t* v,
                 const float* g, const float* beta, int32_t n_req, int32_t W, int32_t init_mode,
                 void* workspace, size_t workspace_bytes, int32_t kernel, dasc_stream_t stream) {
  if (!shape) return DASC_E_INVAL;
  if (!dasc::valid_shape(shape) || shape->dv % 4 != 0) return DASC_E_SHAPE;
  if (layer < 0 || layer >= shape->n_layers || n_req < 1 || W < 1 || W > DASC_MAX_WINDOW ||
      n_pool < 1)
    return DASC_E_INVAL;
  if (init_mode != DASC_INIT_RESTORED && init_mode != DASC_INIT_ZERO) return DASC_E_INVAL;
  if (kernel != DASC_REFRESH_KERNEL_AUTO && kernel != DASC_REFRESH_KERNEL_COLUMN &&
      kernel != DASC_REFRESH_KERNEL_CHANNEL_WY)
    return DASC_E_INVAL;
  if (!inv_row || !states || !slot || !k || !v || !g || !beta) return DASC_E_INVAL;
  if (!dasc::aligned16(states) || !dasc::aligned16(k) || !dasc::aligned16(v)) return DASC_E_INVAL;
  const int dk = shape->dk, dv = shape->dv;
  if (dv > 256) return DASC_E_UNSUPPORTED;
  if (kernel == DASC_REFRESH_KERNEL_CHANNEL_WY && !dasc::refresh_wy_supported(dk, dv))
    return DASC_E_UNSUPPORTED;
  const bool gdn_factors = kernel == DASC_REFRESH_KERNEL_AUTO && uses_gdn_factors(shape);
  const size_t need =
      gdn_factors ? dasc::gdn_factor_workspace_bytes(n_req, shape->n_heads, W) : 0;
  if (workspace_bytes < need || (need > 0 && !workspace)) return DASC_E_WORKSPACE;
  if (need > 0 && !dasc::aligned16(workspace)) return DASC_E_INVAL;
  if (2 * int64_t(n_req) * shape->n_heads > INT32_MAX) return DASC_E_INVAL;  // GDN: 2 blocks a head

  const bool per_channel = shape->arch == DASC_ARCH_KDA;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int zero = init_mode == DASC_INIT_ZERO;
  (void)hipGetLastError();
  if (gdn_factors) {
    if (dasc::gdn_factor_blocks(n_req, shape->n_heads, W) > INT32_MAX) return DASC_E_INVAL;
    dasc::launch_refresh_wy_gdn(n_req, shape->n_heads, shape->n_qk_heads, layer,
                                shape->n_layers, inv_row, states, n_pool, slot, k, v, g, beta, W,
                                zero, workspace, st);
    return dasc::launch_status();
  }
  if (kernel != DASC_REFRESH_KERNEL_COLUMN && dasc::refresh_wy_supported(dk, dv)) {
    dasc::launch_refresh_wy(per_channel, n_req, shape->n_heads, shape->n_qk_heads, layer,
                            shape->n_layers, inv_row, states, n_pool, slot, k, v, g, beta, W,
                            zero, st);
    return dasc::launch_status();
  }
  const int threads = ((dv + 63) / 64) * 64;
  const dim3 grid(unsigned(n_req) * unsigned(shape->n_heads));
  const size_t lds = size_t(kTile) * dv * sizeof(float);
  switch (dk) {
#define DASC_DK(D)                                                                              \
  case D:                                                                                       \
    launch_column<D>(per_channel, grid, dim3(threads), lds, st, shape->n_heads,                 \
                     shape->n_qk_heads, dv, layer, shape->n_layers, inv_row, states, n_pool,    \
                     slot, k, v, g, beta, W, zero);                                             \
    break;
    DASC_DK(16) DASC_DK(32) DASC_DK(64) DASC_DK(128)
#undef DASC_DK
    default: return DASC_E_UNSUPPORTED;
  }
  return dasc::launch_status();
}

}  // namespace dasc

extern "C" int dasc_refresh(const dasc_shape* shape, int32_t layer, const int32_t* inv_row,
                            float* states, int64_t n_pool, const int32_t* slot,
                            const uint16_t* k, const uint16_t* v, const float* g,
                            const float* beta, int32_t n_req, int32_t W, int32_t init_mode,
                            void* workspace, size_t workspace_bytes, dasc_stream_t stream) {
  return dasc::refresh_impl(shape, layer, inv_row, states, n_pool, slot, k, v, g, beta, n_req, W,
                            init_mode, workspace, workspace_bytes, DASC_REFRESH_KERNEL_AUTO,
                            stream);
}

extern "C" int dasc_refresh_select(const dasc_shape* shape, int32_t layer, const int32_t* inv_row,
                                   float* states, int64_t n_pool, const int32_t* slot,
                                   const uint16_t* k, const uint16_t* v, const float* g,
                                   const float* beta, int32_t n_req, int32_t W, int32_t init_mode,
                                   void* workspace, size_t workspace_bytes, int32_t kernel,
                                   dasc_stream_t stream) {
  return dasc::refresh_impl(shape, layer, inv_row, states, n_pool, slot, k, v, g, beta, n_req, W,
                            init_mode, workspace, workspace_bytes, kernel, stream);
}

extern "C" int dasc_restore_refresh(const dasc_shape* shape, int32_t layer, const float* ckpt,
                                    int64_t n_ckpt_slots, const int32_t* src_slot,
                                    int32_t n_ranks, int64_t slice_rows, int64_t n_rows,
                                    const int32_t* inv_row, float* states, int64_t n_pool,
                                    const int32_t* dst_slot, const uint16_t* k,
                                    const uint16_t* v, const float* g, const float* beta,
                                    int32_t n_req, int32_t W, int32_t init_mode,
                                    void* workspace, size_t workspace_bytes,
                                    dasc_stream_t stream) {
  if (!shape) return DASC_E_INVAL;
  if (!dasc::valid_shape(shape) || shape->dv % 4 != 0) return DASC_E_SHAPE;
  if (layer < 0 || layer >= shape->n_layers || n_req < 1 || W < 1 || W > DASC_MAX_WINDOW ||
      n_pool < 1 || n_ckpt_slots < 1 || n_ranks < 1 || n_rows < 0)
    return DASC_E_INVAL;
  if (n_rows > dasc::rows_per_state(shape)) return DASC_E_SHAPE;
  if (n_rows > 0 && (slice_rows < 1 || slice_rows > INT32_MAX || slice_rows * n_ranks < n_rows))
    return DASC_E_INVAL;
  if (init_mode != DASC_INIT_RESTORED && init_mode != DASC_INIT_ZERO) return DASC_E_INVAL;
  if (!inv_row || !states || !src_slot || !dst_slot || !k || !v || !g || !beta)
    return DASC_E_INVAL;
  if (n_rows > 0 && !ckpt) return DASC_E_INVAL;
  if (!dasc::aligned16(states) || !dasc::aligned16(ckpt) || !dasc::aligned16(k) ||
      !dasc::aligned16(v))
    return DASC_E_INVAL;
  size_t need = 0;
  int rc = dasc_refresh_workspace_bytes(shape, n_req, W, &need);
  if (rc != DASC_OK) return rc;
  if (workspace_bytes < need || (need > 0 && !workspace)) return DASC_E_WORKSPACE;
  if (need > 0 && !dasc::aligned16(workspace)) return DASC_E_INVAL;
  if (!dasc::refresh_wy_supported(shape->dk, shape->dv)) return DASC_E_UNSUPPORTED;
  if (2 * int64_t(n_req) * shape->n_heads > INT32_MAX) return DASC_E_INVAL;  // GDN: 2 blocks a head
  if (n_rows == 0) slice_rows = 1;  // nothing is read; keeps the divisor non-zero
  (void)hipGetLastError();
  // GDN heads take the scalar-gate kernel, as in dasc_refresh
  if (uses_gdn_factors(shape)) {
    if (dasc::gdn_factor_blocks(n_req, shape->n_heads, W) > INT32_MAX) return DASC_E_INVAL;
    dasc::launch_restore_refresh_wy_gdn(n_req, shape->n_heads, shape->n_qk_heads, layer,
                                        shape->n_layers, ckpt, n_ckpt_slots, src_slot, slice_rows,
                                        n_rows, inv_row, states, n_pool, dst_slot, k, v, g, beta,
                                        W, init_mode == DASC_INIT_ZERO, workspace,
                                        reinterpret_cast<hipStream_t>(stream));
  } else
    dasc::launch_restore_refresh_wy(shape->arch == DASC_ARCH_KDA, n_req, shape->n_heads,
                                    shape->n_qk_heads, layer, shape->n_layers, ckpt, n_ckpt_slots,
                                    src_slot, slice_rows, n_rows, inv_row, states, n_pool,
                                    dst_slot, k, v, g, beta, W, init_mode == DASC_INIT_ZERO,
                                    reinterpret_cast<hipStream_t>(stream));
  return dasc::launch_status();
}
