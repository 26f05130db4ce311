// Ragged pack (Store) and zero-fill restore (Load) of DASC state checkpoints.
//
// Sec. 4.1 / App. B "Scheme 2": the retained units of all layers are flat-packed,
// layer after layer, into one checkpoint of sum_l r_l units.  Sec. 4.2: on a hit the
// retained units are loaded exactly and the omitted units stay at zero.  Sec. 4.3:
// with T ranks the packed units are cut into slices of C units (one device here).
//
// Both kernels are HBM-bound bit copies.  A state row (one KDA unit, or one of the
// dk rows of a GDN unit) is dv fp32 words = dv/4 128-bit vectors, 512 B at dv = 128.
// A 256-thread block owns a small tile of rows of one checkpoint.  A vector's data
// load depends on its row's index load (unit_row / inv_row), and the two serialise on
// the load counter, so how many reads a CU keeps in flight is set by how many waves
// are resident and by independent loads per thread:
//   pack    one vector per thread (8 rows of 512 B per block), index loaded per lane;
//   restore the block's inv_row entries are staged in LDS first, then every thread
//           issues two independent vector loads.
// Measured on the full-model set (256 checkpoints of 24 x 32 x 128 rows) these beat
// four vectors per thread with per-lane index loads: pack 5.1 -> 6.2 TB/s, restore
// 5.5 -> 5.9 TB/s.  Destination stores are non-temporal: nothing reads a freshly
// written checkpoint or state back from cache.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "dasc.h"
#include "ckpt_layout.h"
#include "launch_common.h"

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kPackUnroll = 1;      // 128-bit vectors per thread
constexpr int kRestoreUnroll = 2;
constexpr int kPackVec = kThreads * kPackUnroll;        // vectors moved per block
constexpr int kRestoreVec = kThreads * kRestoreUnroll;

// VPR_LOG2 >= 0: dv/4 is the power of two 2^VPR_LOG2 (shift/mask addressing).
// VPR_LOG2 <  0: dv/4 given at run time (division addressing).
template <int VPR_LOG2>
struct RowGeom {
  __device__ static int vpr(int) { return 1 << VPR_LOG2; }
  __device__ static int row_of(int v, int) { return v >> VPR_LOG2; }
  __device__ static int col_of(int v, int) { return v & ((1 << VPR_LOG2) - 1); }
};
template <>
struct RowGeom<-1> {
  __device__ static int vpr(int rt) { return rt; }
  __device__ static int row_of(int v, int rt) { return v / rt; }
  __device__ static int col_of(int v, int rt) { return v % rt; }
};

using dasc::slice_row;

// Rows per block: enough 128-bit vectors for every thread to move its share (vec per
// block), or one row when a row alone is longer.
inline int rows_per_block(int vpr, int vec) { return vpr >= vec ? 1 : vec / vpr; }

// A block owns a tile of rows of one rank slice of one checkpoint, so the slice of a
// packed row is known per block and the destination needs no per-row division.
template <int VPR_LOG2>
__device__ __forceinline__ void pack_body(
    const f32x4* __restrict__ states, int64_t n_pool, int64_t rows_state,
    const int32_t* __restrict__ src_slot, const int32_t* __restrict__ unit_row, int64_t n_rows,
    f32x4* __restrict__ ckpt, int64_t n_ckpt_slots, const int32_t* __restrict__ dst_slot,
    int64_t slice_rows, int n_ranks, int blocks_per_slice, int rpb, int vpr_rt,
    const int32_t* __restrict__ slice_begin) {
  using G = RowGeom<VPR_LOG2>;
  const int vpr = G::vpr(vpr_rt);
  // slice-major block order: consecutive blocks fill slice rk of consecutive checkpoint
  // slots, which are adjacent in [T, n_slots, C_rows, dv], so the writes in flight stay
  // in one region instead of spreading over the T slices of one checkpoint
  const int per_slice = int(gridDim.x) / n_ranks;   // n checkpoints x blocks_per_slice
  const int rk = blockIdx.x / per_slice;
  const int rem = blockIdx.x - rk * per_slice;
  const int i = rem / blocks_per_slice;
  const int rb = rem - i * blocks_per_slice;
  const int64_t s = src_slot[i];
  const int64_t d = dst_slot[i];
  if (s < 0 || s >= n_pool || d < 0 || d >= n_ckpt_slots) return;
  const f32x4* src = states + s * rows_state * vpr;
  // Slice rk holds packed rows [slice0, slice_end) at stride slice_rows: equal cuts of
  // the packed rows (rank slices), or, with slice_begin, the layers of the padded layout
  // (rows past the stride are not written).
  const int64_t slice0 = slice_begin ? max(int64_t(slice_begin[rk]), int64_t(0))
                                     : int64_t(rk) * slice_rows;
  const int64_t slice_end = min(min(slice_begin ? int64_t(slice_begin[rk + 1]) : n_rows,
                                    slice0 + slice_rows), n_rows);
  const int64_t row0 = slice0 + int64_t(rb) * rpb;
  // offset of packed row 0 of this slice (may be negative; every row used is >= slice0)
  const int64_t dbase = ((int64_t(rk) * n_ckpt_slots + d) * slice_rows - slice0) * vpr;
  const int n_vec = rpb * vpr;

  for (int base = 0; base < n_vec; base += kPackVec) {
    f32x4 val[kPackUnroll];
    int64_t dst_off[kPackUnroll];
#pragma unroll
    for (int u = 0; u < kPackUnroll; ++u) {
      const int v = base + u * kThreads + threadIdx.x;
      const int64_t j = row0 + G::row_of(v, vpr_rt);
      dst_off[u] = -1;
      if (v < n_vec && j < slice_end) {
        const int64_t dense = unit_row[j];
        if (dense >= 0 && dense < rows_state) {
          const int c = G::col_of(v, vpr_rt);
          val[u] = __builtin_nontemporal_load(src + dense * vpr + c);
          dst_off[u] = j * vpr + c;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kPackUnroll; ++u)
      if (dst_off[u] >= 0) __builtin_nontemporal_store(val[u], ckpt + (dbase + dst_off[u]));
  }
}

template <int VPR_LOG2>
__global__ __launch_bounds__(kThreads) void pack_kernel(
    const f32x4* __restrict__ states, int64_t n_pool, int64_t rows_state,
    const int32_t* __restrict__ src_slot, const int32_t* __restrict__ unit_row, int64_t n_rows,
    f32x4* __restrict__ ckpt, int64_t n_ckpt_slots, const int32_t* __restrict__ dst_slot,
    int64_t slice_rows, int n_ranks, int blocks_per_slice, int rpb, int vpr_rt) {
  pack_body<VPR_LOG2>(states, n_pool, rows_state, src_slot, unit_row, n_rows, ckpt, n_ckpt_slots,
                      dst_slot, slice_rows, n_ranks, blocks_per_slice, rpb, vpr_rt, nullptr);
}

template <int VPR_LOG2>
__global__ __launch_bounds__(kThreads) void pack_padded_kernel(
    const f32x4* __restrict__ states, int64_t n_pool, int64_t rows_state,
    const int32_t* __restrict__ src_slot, const int32_t* __restrict__ unit_row, int64_t n_rows,
    f32x4* __restrict__ ckpt, int64_t n_ckpt_slots, const int32_t* __restrict__ dst_slot,
    int64_t slice_rows, int n_ranks, int blocks_per_slice, int rpb, int vpr_rt,
    const int32_t* __restrict__ slice_begin) {
  pack_body<VPR_LOG2>(states, n_pool, rows_state, src_slot, unit_row, n_rows, ckpt, n_ckpt_slots,
                      dst_slot, slice_rows, n_ranks, blocks_per_slice, rpb, vpr_rt, slice_begin);
}

// Restore body; PADDED selects the padded layout, where the slice of a packed row is
// the layer of its dense row (known per block unless the block straddles two layers).
template <int VPR_LOG2, bool PADDED>
__device__ __forceinline__ void restore_body(
    const f32x4* __restrict__ ckpt, int64_t n_ckpt_slots, const int32_t* __restrict__ src_slot,
    int64_t slice_rows, int64_t n_rows, const int32_t* __restrict__ inv_row,
    f32x4* __restrict__ states, int64_t n_pool, int64_t rows_state,
    const int32_t* __restrict__ dst_slot, int blocks_per_state, int rpb, int vpr_rt,
    const int32_t* __restrict__ slice_begin, int64_t rows_per_layer) {
  using G = RowGeom<VPR_LOG2>;
  const int vpr = G::vpr(vpr_rt);
  const int i = blockIdx.x / blocks_per_state;
  const int rb = blockIdx.x - i * blocks_per_state;
  const int64_t s = src_slot[i];
  const int64_t d = dst_slot[i];
  if (s < 0 || s >= n_ckpt_slots || d < 0 || d >= n_pool) return;
  f32x4* dst = states + d * rows_state * vpr;
  const int64_t row0 = int64_t(rb) * rpb;
  const int n_vec = rpb * vpr;
  // packed index of each row of the tile, read once per row instead of once per lane
  __shared__ int32_t s_inv[kRestoreVec];
  for (int t = threadIdx.x; t < rpb; t += kThreads)
    if (row0 + t < rows_state) s_inv[t] = inv_row[row0 + t];
  __syncthreads();
  int64_t blk_layer = -1;   // padded: the layer of every row of this block, if unique
  if (PADDED) {
    const int64_t last = min(row0 + rpb, rows_state) - 1;
    const int64_t l0 = int64_t(uint32_t(row0) / uint32_t(rows_per_layer));
    if (l0 == int64_t(uint32_t(last) / uint32_t(rows_per_layer))) blk_layer = l0;
  }

  for (int base = 0; base < n_vec; base += kRestoreVec) {
    f32x4 val[kRestoreUnroll];
    int64_t dst_off[kRestoreUnroll];
#pragma unroll
    for (int u = 0; u < kRestoreUnroll; ++u) {
      const int v = base + u * kThreads + threadIdx.x;
      const int r = G::row_of(v, vpr_rt);
      const int64_t dense = row0 + r;
      dst_off[u] = -1;
      val[u] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (v < n_vec && dense < rows_state) {
        const int c = G::col_of(v, vpr_rt);
        const int64_t p = s_inv[r];
        if (p >= 0 && p < n_rows) {
          int64_t row;
          if (PADDED) {
            const int64_t l = blk_layer >= 0 ? blk_layer
                                             : int64_t(uint32_t(dense) / uint32_t(rows_per_layer));
            const int64_t e = p - slice_begin[l];
            row = (e >= 0 && e < slice_rows) ? (l * n_ckpt_slots + s) * slice_rows + e : -1;
          } else {
            row = slice_row(p, slice_rows, n_rows, n_ckpt_slots, s);
          }
          if (row >= 0) val[u] = __builtin_nontemporal_load(ckpt + row * vpr + c);
        }
        dst_off[u] = dense * vpr + c;
      }
    }
#pragma unroll
    for (int u = 0; u < kRestoreUnroll; ++u)
      if (dst_off[u] >= 0) __builtin_nontemporal_store(val[u], dst + dst_off[u]);
  }
}

template <int VPR_LOG2>
__global__ __launch_bounds__(kThreads) void restore_kernel(
    const f32x4* __restrict__ ckpt, int64_t n_ckpt_slots, const int32_t* __restrict__ src_slot,
    int64_t slice_rows, int64_t n_rows, const int32_t* __restrict__ inv_row,
    f32x4* __restrict__ states, int64_t n_pool, int64_t rows_state,
    const int32_t* __restrict__ dst_slot, int blocks_per_state, int rpb, int vpr_rt) {
  restore_body<VPR_LOG2, false>(ckpt, n_ckpt_slots, src_slot, slice_rows, n_rows, inv_row, states,
                                n_pool, rows_state, dst_slot, blocks_per_state, rpb, vpr_rt,
                                nullptr, 1);
}

template <int VPR_LOG2>
__global__ __launch_bounds__(kThreads) void restore_padded_kernel(
    const f32x4* __restrict__ ckpt, int64_t n_ckpt_slots, const int32_t* __restrict__ src_slot,
    int64_t slice_rows, int64_t n_rows, const int32_t* __restrict__ inv_row,
    f32x4* __restrict__ states, int64_t n_pool, int64_t rows_state,
    const int32_t* __restrict__ dst_slot, int blocks_per_state, int rpb, int vpr_rt,
    const int32_t* __restrict__ slice_begin, int64_t rows_per_layer) {
  restore_body<VPR_LOG2, true>(ckpt, n_ckpt_slots, src_slot, slice_rows, n_rows, inv_row, states,
                               n_pool, rows_state, dst_slot, blocks_per_state, rpb, vpr_rt,
                               slice_begin, rows_per_layer);
}

int vpr_log2(int vpr) {
  for (int l = 0; l <= 8; ++l)
    if (vpr == (1 << l)) return l;
  return -1;
}

#define DASC_LAUNCH_BY_VPR(KERNEL, lg, grid, st, ...)                                   \
  switch (lg) {                                                                         \
    case 0: hipLaunchKernelGGL(KERNEL<0>, grid, dim3(kThreads), 0, st, __VA_ARGS__); break; \
    case 1: hipLaunchKernelGGL(KERNEL<1>, grid, dim3(kThreads), 0, st, __VA_ARGS__); break; \
    case 2: hipLaunchKernelGGL(KERNEL<2>, grid, dim3(kThreads), 0, st, __VA_ARGS__); break; \
    case 3: hipLaunchKernelGGL(KERNEL<3>, grid, dim3(kThreads), 0, st, __VA_ARGS__); break; \
    case 4: hipLaunchKernelGGL(KERNEL<4>, grid, dim3(kThreads), 0, st, __VA_ARGS__); break; \
    case 5: hipLaunchKernelGGL(KERNEL<5>, grid, dim3(kThreads), 0, st, __VA_ARGS__); break; \
    case 6: hipLaunchKernelGGL(KERNEL<6>, grid, dim3(kThreads), 0, st, __VA_ARGS__); break; \
    case 7: hipLaunchKernelGGL(KERNEL<7>, grid, dim3(kThreads), 0, st, __VA_ARGS__); break; \
    case 8: hipLaunchKernelGGL(KERNEL<8>, grid, dim3(kThreads), 0, st, __VA_ARGS__); break; \
    default: hipLaunchKernelGGL(KERNEL<-1>, grid, dim3(kThreads), 0, st, __VA_ARGS__); break; \
  }

int check_common(const dasc_shape* shape, int64_t n_pool, int64_t n_ckpt_slots, int32_t n_ranks,
                 int64_t slice_rows, int64_t n_rows, int32_t n) {
  if (!dasc::valid_shape(shape)) return DASC_E_SHAPE;
  if (shape->dv % 4 != 0) return DASC_E_SHAPE;
  if (n < 0 || n_pool < 1 || n_ckpt_slots < 1 || n_ranks < 1 || n_rows < 0) return DASC_E_INVAL;
  if (n_rows > dasc::rows_per_state(shape)) return DASC_E_SHAPE;
  if (n_rows > 0 && (slice_rows < 1 || slice_rows > INT32_MAX || slice_rows * n_ranks < n_rows))
    return DASC_E_INVAL;
  return DASC_OK;
}

}  // namespace

extern "C" int dasc_pack(const dasc_shape* shape, const float* states, int64_t n_pool,
                         const int32_t* src_slot, const int32_t* unit_row, int64_t n_rows,
                         float* ckpt, int64_t n_ckpt_slots, const int32_t* dst_slot,
                         int32_t n_ranks, int64_t slice_rows, int32_t n, dasc_stream_t stream) {
  int rc = check_common(shape, n_pool, n_ckpt_slots, n_ranks, slice_rows, n_rows, n);
  if (rc != DASC_OK) return rc;
  if (n == 0 || n_rows == 0) return DASC_OK;
  if (!states || !src_slot || !unit_row || !ckpt || !dst_slot) return DASC_E_INVAL;
  if (!dasc::aligned16(states) || !dasc::aligned16(ckpt)) return DASC_E_INVAL;
  const int vpr = shape->dv / 4;
  const int rpb = rows_per_block(vpr, kPackVec);
  // blocks per rank slice: a slice holds at most min(slice_rows, n_rows) packed rows
  const int64_t bps = (std::min<int64_t>(slice_rows, n_rows) + rpb - 1) / rpb;
  const int64_t blocks = bps * n_ranks * n;
  if (blocks > INT32_MAX) return DASC_E_INVAL;
  (void)hipGetLastError();
  DASC_LAUNCH_BY_VPR(pack_kernel, vpr_log2(vpr), dim3(unsigned(blocks)),
                     reinterpret_cast<hipStream_t>(stream),
                     reinterpret_cast<const f32x4*>(states), n_pool, dasc::rows_per_state(shape),
                     src_slot, unit_row, n_rows, reinterpret_cast<f32x4*>(ckpt), n_ckpt_slots,
                     dst_slot, slice_rows, int(n_ranks), int(bps), rpb, vpr);
  return dasc::launch_status();
}

extern "C" int dasc_restore(const dasc_shape* shape, const float* ckpt, int64_t n_ckpt_slots,
                            const int32_t* src_slot, int32_t n_ranks, int64_t slice_rows,
                            int64_t n_rows, const int32_t* inv_row, float* states,
                            int64_t n_pool, const int32_t* dst_slot, int32_t n,
                            dasc_stream_t stream) {
  int rc = check_common(shape, n_pool, n_ckpt_slots, n_ranks, slice_rows, n_rows, n);
  if (rc != DASC_OK) return rc;
  if (n == 0) return DASC_OK;
  if (!src_slot || !inv_row || !states || !dst_slot) return DASC_E_INVAL;
  if (n_rows > 0 && !ckpt) return DASC_E_INVAL;
  if (!dasc::aligned16(states) || !dasc::aligned16(ckpt)) return DASC_E_INVAL;
  if (n_rows == 0) slice_rows = 1;  // nothing is read; keeps the divisor non-zero
  const int vpr = shape->dv / 4;
  const int rpb = rows_per_block(vpr, kRestoreVec);
  const int64_t rows = dasc::rows_per_state(shape);
  const int64_t bps = (rows + rpb - 1) / rpb;
  if (bps * n > INT32_MAX) return DASC_E_INVAL;
  (void)hipGetLastError();
  DASC_LAUNCH_BY_VPR(restore_kernel, vpr_log2(vpr), dim3(unsigned(bps * n)),
                     reinterpret_cast<hipStream_t>(stream),
                     reinterpret_cast<const f32x4*>(ckpt), n_ckpt_slots, src_slot, slice_rows,
                     n_rows, inv_row, reinterpret_cast<f32x4*>(states), n_pool, rows, dst_slot,
                     int(bps), rpb, vpr);
  return dasc::launch_status();
}

// ---- App. B Scheme 1: padded layout [L, n_slots, r_max_rows, dv] ---------------------
// The rank-slice kernels with one slice per layer: slice l starts at packed row
// layer_off_rows[l] and is stored at stride r_max_rows.

extern "C" int dasc_pack_padded(const dasc_shape* shape, const float* states, int64_t n_pool,
                                const int32_t* src_slot, const int32_t* unit_row,
                                int64_t n_rows, const int32_t* layer_off_rows,
                                int64_t r_max_rows, float* ckpt, int64_t n_ckpt_slots,
                                const int32_t* dst_slot, int32_t n, dasc_stream_t stream) {
  int rc = check_common(shape, n_pool, n_ckpt_slots, 1, n_rows, n_rows, n);
  if (rc != DASC_OK) return rc;
  if (r_max_rows < 0 || r_max_rows > INT32_MAX || (n_rows > 0 && r_max_rows < 1))
    return DASC_E_INVAL;
  if (n == 0 || n_rows == 0) return DASC_OK;
  if (!states || !src_slot || !unit_row || !layer_off_rows || !ckpt || !dst_slot)
    return DASC_E_INVAL;
  if (!dasc::aligned16(states) || !dasc::aligned16(ckpt)) return DASC_E_INVAL;
  const int L = shape->n_layers;
  const int vpr = shape->dv / 4;
  const int rpb = rows_per_block(vpr, kPackVec);
  const int64_t bps = (std::min<int64_t>(r_max_rows, n_rows) + rpb - 1) / rpb;
  const int64_t blocks = bps * L * n;
  if (blocks > INT32_MAX) return DASC_E_INVAL;
  (void)hipGetLastError();
  DASC_LAUNCH_BY_VPR(pack_padded_kernel, vpr_log2(vpr), dim3(unsigned(blocks)),
                     reinterpret_cast<hipStream_t>(stream),
                     reinterpret_cast<const f32x4*>(states), n_pool, dasc::rows_per_state(shape),
                     src_slot, unit_row, n_rows, reinterpret_cast<f32x4*>(ckpt), n_ckpt_slots,
                     dst_slot, r_max_rows, L, int(bps), rpb, vpr, layer_off_rows);
  return dasc::launch_status();
}

extern "C" int dasc_restore_padded(const dasc_shape* shape, const float* ckpt,
                                   int64_t n_ckpt_slots, const int32_t* src_slot,
                                   const int32_t* layer_off_rows, int64_t r_max_rows,
                                   int64_t n_rows, const int32_t* inv_row, float* states,
                                   int64_t n_pool, const int32_t* dst_slot, int32_t n,
                                   dasc_stream_t stream) {
  int rc = check_common(shape, n_pool, n_ckpt_slots, 1, n_rows, n_rows, n);
  if (rc != DASC_OK) return rc;
  if (r_max_rows < 0 || r_max_rows > INT32_MAX || (n_rows > 0 && r_max_rows < 1))
    return DASC_E_INVAL;
  if (n == 0) return DASC_OK;
  if (!src_slot || !inv_row || !states || !dst_slot) return DASC_E_INVAL;
  if (n_rows > 0 && (!ckpt || !layer_off_rows)) return DASC_E_INVAL;
  if (!dasc::aligned16(states) || !dasc::aligned16(ckpt)) return DASC_E_INVAL;
  if (n_rows == 0) r_max_rows = 1;  // nothing is read
  const int vpr = shape->dv / 4;
  const int rpb = rows_per_block(vpr, kRestoreVec);
  const int64_t rows = dasc::rows_per_state(shape);
  const int64_t bps = (rows + rpb - 1) / rpb;
  if (bps * n > INT32_MAX) return DASC_E_INVAL;
  (void)hipGetLastError();
  DASC_LAUNCH_BY_VPR(restore_padded_kernel, vpr_log2(vpr), dim3(unsigned(bps * n)),
                     reinterpret_cast<hipStream_t>(stream),
                     reinterpret_cast<const f32x4*>(ckpt), n_ckpt_slots, src_slot, r_max_rows,
                     n_rows, inv_row, reinterpret_cast<f32x4*>(states), n_pool, rows, dst_slot,
                     int(bps), rpb, vpr, n_rows > 0 ? layer_off_rows : nullptr,
                     int64_t(shape->n_heads) * shape->dk);
  return dasc::launch_status();
}
