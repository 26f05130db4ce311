// Internal launchers of the refresh kernels (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "dasc.h"

namespace dasc {

// The body of dasc_refresh with an explicit kernel choice (DASC_REFRESH_KERNEL_*, see
// dasc_testing.h); validates every argument before it launches anything.
int refresh_impl(const dasc_shape* shape, int32_t layer, const int32_t* inv_row, float* states,
                 int64_t n_pool, const int32_t* slot, const uint16_t* k, const uint16_t* v,
                 const float* g, const float* beta, int32_t n_req, int32_t W, int32_t init_mode,
                 void* workspace, size_t workspace_bytes, int32_t kernel, dasc_stream_t stream);

// Chunkwise WY-form kernel on bf16 MFMA; built for dk = dv = 128 only.
bool refresh_wy_supported(int dk, int dv);
void launch_refresh_wy(bool per_channel, int n_req, int H, int Hqk, int layer, int L,
                       const int32_t* inv_row, float* states, int64_t n_pool, const int32_t* slot,
                       const uint16_t* k, const uint16_t* v, const float* g, const float* beta,
                       int W, int init_zero, hipStream_t st);

// GDN heads (scalar gate per token), dk = dv = 128: keys enter the MFMAs exactly and
// the decays stay outside the contractions.  Two launches: the per-chunk factor -T' of
// every refreshed head into `ws`, then the state recurrence (two blocks per head, one per
// value-column half) reading it.  `ws` holds gdn_factor_workspace_bytes(n_req, H, W).
constexpr int kGdnFactorBytesPerChunk = 4096;
size_t gdn_factor_workspace_bytes(int n_req, int H, int W);
int64_t gdn_factor_blocks(int n_req, int H, int W);
void launch_refresh_wy_gdn(int n_req, int H, int Hqk, int layer, int L, const int32_t* inv_row,
                           float* states, int64_t n_pool, const int32_t* slot, const uint16_t* k,
                           const uint16_t* v, const float* g, const float* beta, int W,
                           int init_zero, void* ws, hipStream_t st);

// The same kernel fused with the restore of the layer: the initial state of each head is
// read from the packed checkpoint (kept rows; omitted rows start at zero) and every row
// of the layer is written (omitted rows refreshed, kept rows copied bit for bit).
void launch_restore_refresh_wy(bool per_channel, int n_req, int H, int Hqk, int layer, int L,
                               const float* ckpt, int64_t n_ckpt_slots, const int32_t* ck_slot,
                               int64_t slice_rows, int64_t n_rows, const int32_t* inv_row,
                               float* states, int64_t n_pool, const int32_t* slot,
                               const uint16_t* k, const uint16_t* v, const float* g,
                               const float* beta, int W, int init_zero, hipStream_t st);

// The scalar-gate GDN kernel's fused variant (dk = dv = 128).
void launch_restore_refresh_wy_gdn(int n_req, int H, int Hqk, int layer, int L, const float* ckpt,
                                   int64_t n_ckpt_slots, const int32_t* ck_slot,
                                   int64_t slice_rows, int64_t n_rows, const int32_t* inv_row,
                                   float* states, int64_t n_pool, const int32_t* slot,
                                   const uint16_t* k, const uint16_t* v, const float* g,
                                   const float* beta, int W, int init_zero, void* ws,
                                   hipStream_t st);

}  // namespace dasc
