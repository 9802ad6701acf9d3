// Host-side launchers of the SBVR kernels (internal to libsbvr).  Arguments
// are validated by the C ABI layer before these are called; each returns an
// sbvr_status and enqueues work on `stream` only.
#pragma once

#include <hip/hip_runtime.h>

#include "layout.h"
#include "sbvr.h"

namespace sbvr {

// Dynamic LDS per workgroup that a launch may request without raising the
// kernel's attribute; launch shapes are capped to stay within it.
constexpr size_t SBVR_MAX_DYN_LDS = 64 * 1024;

inline int launch_kernel(const void *fn, dim3 grid, dim3 block, size_t lds, hipStream_t stream,
                         void **args)
{
    return hipLaunchKernel(fn, grid, block, args, lds, stream) == hipSuccess ? SBVR_OK : SBVR_E_HIP;
}

int launch_pack(const Dims &d, const uint32_t *planes_canon, const uint16_t *coeffs_canon,
                void *planes_dev, void *coeffs_dev, hipStream_t stream);
int launch_unpack(const Dims &d, const void *planes_dev, const void *coeffs_dev,
                  uint32_t *planes_canon, uint16_t *coeffs_canon, hipStream_t stream);
// Device weights: planes plus either per-group coefficient blocks (index ==
// nullptr) or the coefficient-cache format (index blocks + table of n_sets
// coefficient sets).
struct WeightRef {
    const void *planes;
    const void *coeffs;
    const void *index;
    const void *table;
    int n_sets;
};

inline WeightRef per_group_weights(const void *planes, const void *coeffs)
{
    return WeightRef{planes, coeffs, nullptr, nullptr, 0};
}

// a8: activations converted online to SBVR-8 (the W4A8 decode path)
int launch_gemv_b1(const Dims &d, const WeightRef &w, const uint16_t *x, uint16_t *y, bool a8,
                   hipStream_t stream);
int launch_gemv_b1s(const Dims &d, const WeightRef &w, const uint16_t *x, uint16_t *y, bool a8,
                    hipStream_t stream);
int launch_pack_indexed(const Dims &d, int n_sets, const uint32_t *planes_canon, const uint16_t *index_canon,
                        const uint16_t *table_canon, void *planes_dev, void *index_dev, void *table_dev,
                        hipStream_t stream);
int launch_unpack_indexed(const Dims &d, int n_sets, const void *planes_dev, const void *index_dev,
                          const void *table_dev, uint32_t *planes_canon, uint16_t *index_canon,
                          uint16_t *table_canon, hipStream_t stream);
int launch_decompress(const Dims &d, const WeightRef &w, uint16_t *W, hipStream_t stream);
int launch_encode(int O, int I, int k, const float *W, int n_ratio1, int n_ratio2, int n_scale, int n_bias,
                  int normalise, uint32_t *planes, uint16_t *coeffs, double *mse, hipStream_t stream);
int launch_encode_cached(int O, int I, int k, const float *W, int n_ratio1, int n_ratio2, int n_scale, int n_bias,
                         int normalise, int slots, uint32_t *planes, uint16_t *coeffs, double *mse, uint8_t *hits,
                         hipStream_t stream);
int launch_prefill(const Dims &d, const void *planes_dev, const void *coeffs_dev, const uint16_t *X, uint16_t *Y,
                   int T, hipStream_t stream);
int launch_gemm_sbs(const Dims &d, const void *planes_dev, const void *coeffs_dev,
                    const uint16_t *X, uint16_t *Y, int B, hipStream_t stream);

// Grouped batch-1 GEMV: n (<= GROUP_MAX) matrices with the same I and k, each
// with its own weights (per-group coefficients), binary16 activations and
// output, in one launch.  The launch shape is the one a single matrix with
// all the members' row tiles would get; every member's row tiles start a new
// workgroup.
struct GemvMember {
    int O;
    const void *planes;
    const void *coeffs;
    const uint16_t *x;
    uint16_t *y;
};
struct GemvGroup;
// Fills the member table for workgroups of `tiles_per_group` row tiles and
// returns the grid size.
int fill_group(GemvGroup &g, int n, const GemvMember *mem, const Dims &d, int tiles_per_group);
// a8: activations converted online to SBVR-8 (every member)
int launch_gemv_group(int n, const GemvMember *mem, int I, int k, bool a8, hipStream_t stream);
int launch_gemv_b1s_group(const Dims &d, int n, const GemvMember *mem, bool a8, hipStream_t stream);

}  // namespace sbvr
