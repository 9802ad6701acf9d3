// C ABI of libsbvr (include/sbvr.h): argument validation, then dispatch to the
// kernel launchers.  Validation happens entirely on the host before any HIP
// call, so a rejected call enqueues nothing and touches no output.
#include <stdint.h>

#include "launch.h"
#include "sbvr.h"

using namespace sbvr;

namespace {

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

int check_shape(int O, int I, int k)
{
    if (O < 1 || I < GROUP || I % GROUP != 0 || k < 1)
        return SBVR_E_INVALID_ARG;
    if (k > MAX_K)
        return SBVR_E_UNSUPPORTED;
    // element offsets inside the kernels are 32-bit
    if ((long long)O * I > (1ll << 31) - 1)
        return SBVR_E_UNSUPPORTED;
    // byte offsets within a workgroup's range of tiles are 32-bit and must stay
    // below the per-lane "read zero" offset (2^30): one tile's plane bytes over
    // all gblocks (n_gblocks * GB * TR * k * 16) are capped at 2^26, i.e.
    // I <= 2^25 at k = 4 (the activation offsets of a row then fit an int too)
    const Dims d = make_dims(O, I, k);
    if ((long long)d.n_gblocks * GB * d.tr * k * 16 > (1ll << 26))
        return SBVR_E_UNSUPPORTED;
    return SBVR_OK;
}

int check_repack(int O, int I, int k, const void *planes_canon, const void *coeffs_canon,
                 const void *planes_dev, const void *coeffs_dev)
{
    int st = check_shape(O, I, k);
    if (st != SBVR_OK)
        return st;
    if (!planes_canon || !coeffs_canon || !planes_dev || !coeffs_dev)
        return SBVR_E_INVALID_ARG;
    if (!aligned(planes_canon, 16) || !aligned(coeffs_canon, 2) || !aligned(planes_dev, 16) ||
        !aligned(coeffs_dev, 16))
        return SBVR_E_ALIGNMENT;
    return SBVR_OK;
}

int check_gemv(int O, int I, int k, const void *planes_dev, const void *coeffs_dev,
               const uint16_t *x, const uint16_t *y, int B, size_t ws_bytes)
{
    int st = check_shape(O, I, k);
    if (st != SBVR_OK)
        return st;
    if (B < 1 || B > 8)
        return SBVR_E_INVALID_ARG;
    if (!planes_dev || !coeffs_dev || !x || !y)
        return SBVR_E_INVALID_ARG;
    if (!aligned(planes_dev, 16) || !aligned(coeffs_dev, 16) || !aligned(x, 16) || !aligned(y, 2))
        return SBVR_E_ALIGNMENT;
    if (ws_bytes < sbvr_workspace_bytes(O, I, k, B))
        return SBVR_E_WORKSPACE;
    return SBVR_OK;
}

int check_sets(int n_sets) { return n_sets >= 1 && n_sets <= MAX_SETS ? SBVR_OK : SBVR_E_INVALID_ARG; }

int check_indexed_gemv(int O, int I, int k, int n_sets, const void *planes_dev, const void *index_dev,
                       const void *table_dev, const uint16_t *x, const uint16_t *y, size_t ws_bytes)
{
    int st = check_shape(O, I, k);
    if (st != SBVR_OK)
        return st;
    if ((st = check_sets(n_sets)) != SBVR_OK)
        return st;
    if (!planes_dev || !index_dev || !table_dev || !x || !y)
        return SBVR_E_INVALID_ARG;
    if (!aligned(planes_dev, 16) || !aligned(index_dev, 16) || !aligned(table_dev, 16) || !aligned(x, 16) ||
        !aligned(y, 2))
        return SBVR_E_ALIGNMENT;
    if (ws_bytes < sbvr_workspace_bytes(O, I, k, 1))
        return SBVR_E_WORKSPACE;
    return SBVR_OK;
}

int check_indexed_repack(int O, int I, int k, int n_sets, const void *planes_canon, const void *index_canon,
                         const void *table_canon, const void *planes_dev, const void *index_dev,
                         const void *table_dev)
{
    int st = check_shape(O, I, k);
    if (st != SBVR_OK)
        return st;
    if ((st = check_sets(n_sets)) != SBVR_OK)
        return st;
    if (!planes_canon || !index_canon || !table_canon || !planes_dev || !index_dev || !table_dev)
        return SBVR_E_INVALID_ARG;
    if (!aligned(planes_canon, 16) || !aligned(index_canon, 2) || !aligned(table_canon, 2) ||
        !aligned(planes_dev, 16) || !aligned(index_dev, 16) || !aligned(table_dev, 16))
        return SBVR_E_ALIGNMENT;
    return SBVR_OK;
}

WeightRef indexed_weights(const void *planes, const void *index, const void *table, int n_sets)
{
    return WeightRef{planes, nullptr, index, table, n_sets};
}

int grouped_gemv(int n, const int *O, int I, int k, const void *const *planes_dev, const void *const *coeffs_dev,
                 const uint16_t *const *x, uint16_t *const *y, size_t ws_bytes, bool a8, hipStream_t stream)
{
    if (n < 1 || n > SBVR_GEMV_GROUP_MAX || !O || !planes_dev || !coeffs_dev || !x || !y)
        return SBVR_E_INVALID_ARG;
    GemvMember mem[SBVR_GEMV_GROUP_MAX];
    for (int i = 0; i < n; ++i) {
        int st = check_gemv(O[i], I, k, planes_dev[i], coeffs_dev[i], x[i], y[i], 1, ws_bytes);
        if (st != SBVR_OK)
            return st;
        mem[i] = GemvMember{O[i], planes_dev[i], coeffs_dev[i], x[i], y[i]};
    }
    return launch_gemv_group(n, mem, I, k, a8, stream);
}

}  // namespace

extern "C" {

const char *sbvr_status_string(int status)
{
    switch (status) {
    case SBVR_OK: return "SBVR_OK";
    case SBVR_E_INVALID_ARG: return "SBVR_E_INVALID_ARG";
    case SBVR_E_UNSUPPORTED: return "SBVR_E_UNSUPPORTED";
    case SBVR_E_WORKSPACE: return "SBVR_E_WORKSPACE";
    case SBVR_E_ALIGNMENT: return "SBVR_E_ALIGNMENT";
    case SBVR_E_HIP: return "SBVR_E_HIP";
    default: return "SBVR_E_UNKNOWN";
    }
}

int sbvr_version(void) { return 107; }

size_t sbvr_packed_plane_bytes(int O, int I, int k)
{
    return check_shape(O, I, k) == SBVR_OK ? plane_bytes(make_dims(O, I, k)) : 0;
}

size_t sbvr_packed_coeff_bytes(int O, int I, int k)
{
    return check_shape(O, I, k) == SBVR_OK ? coeff_bytes(make_dims(O, I, k)) : 0;
}

size_t sbvr_workspace_bytes(int O, int I, int k, int B)
{
    (void)O;
    (void)I;
    (void)k;
    (void)B;
    return 0;
}

int sbvr_pack(int O, int I, int k, const uint32_t *planes_canon, const uint16_t *coeffs_canon,
              void *planes_dev, void *coeffs_dev, hipStream_t stream)
{
    int st = check_repack(O, I, k, planes_canon, coeffs_canon, planes_dev, coeffs_dev);
    if (st != SBVR_OK)
        return st;
    return launch_pack(make_dims(O, I, k), planes_canon, coeffs_canon, planes_dev, coeffs_dev, stream);
}

int sbvr_unpack(int O, int I, int k, const void *planes_dev, const void *coeffs_dev,
                uint32_t *planes_canon, uint16_t *coeffs_canon, hipStream_t stream)
{
    int st = check_repack(O, I, k, planes_canon, coeffs_canon, planes_dev, coeffs_dev);
    if (st != SBVR_OK)
        return st;
    return launch_unpack(make_dims(O, I, k), planes_dev, coeffs_dev, planes_canon, coeffs_canon, stream);
}

int sbvr_gemv(int O, int I, int k, const void *planes_dev, const void *coeffs_dev,
              const uint16_t *x, uint16_t *y, void *workspace, size_t ws_bytes, hipStream_t stream)
{
    (void)workspace;
    int st = check_gemv(O, I, k, planes_dev, coeffs_dev, x, y, 1, ws_bytes);
    if (st != SBVR_OK)
        return st;
    return launch_gemv_b1(make_dims(O, I, k), per_group_weights(planes_dev, coeffs_dev), x, y, false, stream);
}

int sbvr_gemm_small_batch(int O, int I, int k, const void *planes_dev, const void *coeffs_dev,
                          const uint16_t *X, uint16_t *Y, int B, void *workspace, size_t ws_bytes,
                          hipStream_t stream)
{
    (void)workspace;
    int st = check_gemv(O, I, k, planes_dev, coeffs_dev, X, Y, B, ws_bytes);
    if (st != SBVR_OK)
        return st;
    const Dims d = make_dims(O, I, k);
    if (B == 1)
        return launch_gemv_b1(d, per_group_weights(planes_dev, coeffs_dev), X, Y, false, stream);
    return launch_gemm_sbs(d, planes_dev, coeffs_dev, X, Y, B, stream);
}

int sbvr_gemv_a8(int O, int I, int k, const void *planes_dev, const void *coeffs_dev,
                 const uint16_t *x, uint16_t *y, void *workspace, size_t ws_bytes, hipStream_t stream)
{
    (void)workspace;
    int st = check_gemv(O, I, k, planes_dev, coeffs_dev, x, y, 1, ws_bytes);
    if (st != SBVR_OK)
        return st;
    return launch_gemv_b1(make_dims(O, I, k), per_group_weights(planes_dev, coeffs_dev), x, y, true, stream);
}


int sbvr_gemv_grouped(int n, const int *O, int I, int k, const void *const *planes_dev,
                      const void *const *coeffs_dev, const uint16_t *const *x, uint16_t *const *y,
                      void *workspace, size_t ws_bytes, hipStream_t stream)
{
    (void)workspace;
    return grouped_gemv(n, O, I, k, planes_dev, coeffs_dev, x, y, ws_bytes, false, stream);
}

int sbvr_gemv_grouped_a8(int n, const int *O, int I, int k, const void *const *planes_dev,
                         const void *const *coeffs_dev, const uint16_t *const *x, uint16_t *const *y,
                         void *workspace, size_t ws_bytes, hipStream_t stream)
{
    (void)workspace;
    return grouped_gemv(n, O, I, k, planes_dev, coeffs_dev, x, y, ws_bytes, true, stream);
}

size_t sbvr_packed_index_bytes(int O, int I, int k)
{
    return check_shape(O, I, k) == SBVR_OK ? index_bytes(make_dims(O, I, k)) : 0;
}

size_t sbvr_packed_table_bytes(int n_sets, int k)
{
    return check_sets(n_sets) == SBVR_OK && k >= 1 && k <= MAX_K ? table_bytes(n_sets) : 0;
}

int sbvr_pack_indexed(int O, int I, int k, int n_sets, const uint32_t *planes_canon,
                      const uint16_t *index_canon, const uint16_t *table_canon, void *planes_dev,
                      void *index_dev, void *table_dev, hipStream_t stream)
{
    int st = check_indexed_repack(O, I, k, n_sets, planes_canon, index_canon, table_canon, planes_dev,
                                  index_dev, table_dev);
    if (st != SBVR_OK)
        return st;
    return launch_pack_indexed(make_dims(O, I, k), n_sets, planes_canon, index_canon, table_canon,
                               planes_dev, index_dev, table_dev, stream);
}

int sbvr_unpack_indexed(int O, int I, int k, int n_sets, const void *planes_dev, const void *index_dev,
                        const void *table_dev, uint32_t *planes_canon, uint16_t *index_canon,
                        uint16_t *table_canon, hipStream_t stream)
{
    int st = check_indexed_repack(O, I, k, n_sets, planes_canon, index_canon, table_canon, planes_dev,
                                  index_dev, table_dev);
    if (st != SBVR_OK)
        return st;
    return launch_unpack_indexed(make_dims(O, I, k), n_sets, planes_dev, index_dev, table_dev, planes_canon,
                                 index_canon, table_canon, stream);
}

int sbvr_gemv_indexed(int O, int I, int k, int n_sets, const void *planes_dev, const void *index_dev,
                      const void *table_dev, const uint16_t *x, uint16_t *y, void *workspace,
                      size_t ws_bytes, hipStream_t stream)
{
    (void)workspace;
    int st = check_indexed_gemv(O, I, k, n_sets, planes_dev, index_dev, table_dev, x, y, ws_bytes);
    if (st != SBVR_OK)
        return st;
    return launch_gemv_b1(make_dims(O, I, k), indexed_weights(planes_dev, index_dev, table_dev, n_sets), x, y,
                          false, stream);
}

int sbvr_gemv_indexed_a8(int O, int I, int k, int n_sets, const void *planes_dev, const void *index_dev,
                         const void *table_dev, const uint16_t *x, uint16_t *y, void *workspace,
                         size_t ws_bytes, hipStream_t stream)
{
    (void)workspace;
    int st = check_indexed_gemv(O, I, k, n_sets, planes_dev, index_dev, table_dev, x, y, ws_bytes);
    if (st != SBVR_OK)
        return st;
    return launch_gemv_b1(make_dims(O, I, k), indexed_weights(planes_dev, index_dev, table_dev, n_sets), x, y,
                          true, stream);
}

namespace {
int check_encode(int O, int I, int k, const float *W, int n_ratio1, int n_ratio2, int n_scale, int n_bias,
                 int normalise, uint32_t *planes_canon, uint16_t *coeffs_canon, double *mse)
{
    int st = check_shape(O, I, k);
    if (st != SBVR_OK)
        return st;
    if (n_ratio1 < 1 || n_ratio2 < 1 || n_scale < 1 || n_bias < 1 || (normalise != 0 && normalise != 1))
        return SBVR_E_INVALID_ARG;
    if ((long long)(n_ratio1 + (long long)n_ratio2) * n_scale * n_bias > SBVR_ENCODE_MAX_ENTRIES)
        return SBVR_E_UNSUPPORTED;
    if (!W || !planes_canon || !coeffs_canon)
        return SBVR_E_INVALID_ARG;
    if (!aligned(W, 4) || !aligned(planes_canon, 16) || !aligned(coeffs_canon, 2) || (mse && !aligned(mse, 8)))
        return SBVR_E_ALIGNMENT;
    return SBVR_OK;
}
}  // namespace

int sbvr_encode(int O, int I, int k, const float *W, int n_ratio1, int n_ratio2, int n_scale, int n_bias,
                int normalise, uint32_t *planes_canon, uint16_t *coeffs_canon, double *mse, hipStream_t stream)
{
    int st = check_encode(O, I, k, W, n_ratio1, n_ratio2, n_scale, n_bias, normalise, planes_canon, coeffs_canon,
                          mse);
    if (st != SBVR_OK)
        return st;
    return launch_encode(O, I, k, W, n_ratio1, n_ratio2, n_scale, n_bias, normalise, planes_canon, coeffs_canon,
                         mse, stream);
}

int sbvr_encode_cached(int O, int I, int k, const float *W, int n_ratio1, int n_ratio2, int n_scale, int n_bias,
                       int normalise, int cache_slots, uint32_t *planes_canon, uint16_t *coeffs_canon, double *mse,
                       uint8_t *hits, hipStream_t stream)
{
    int st = check_encode(O, I, k, W, n_ratio1, n_ratio2, n_scale, n_bias, normalise, planes_canon, coeffs_canon,
                          mse);
    if (st != SBVR_OK)
        return st;
    if (cache_slots < 0 || cache_slots > SBVR_ENCODE_CACHE_MAX)
        return SBVR_E_INVALID_ARG;
    return launch_encode_cached(O, I, k, W, n_ratio1, n_ratio2, n_scale, n_bias, normalise, cache_slots,
                                planes_canon, coeffs_canon, mse, hits, stream);
}

int sbvr_decompress(int O, int I, int k, const void *planes_dev, const void *coeffs_dev, uint16_t *W,
                    hipStream_t stream)
{
    int st = check_shape(O, I, k);
    if (st != SBVR_OK)
        return st;
    if (!planes_dev || !coeffs_dev || !W)
        return SBVR_E_INVALID_ARG;
    if (!aligned(planes_dev, 16) || !aligned(coeffs_dev, 16) || !aligned(W, 16))
        return SBVR_E_ALIGNMENT;
    return launch_decompress(make_dims(O, I, k), per_group_weights(planes_dev, coeffs_dev), W, stream);
}

int sbvr_gemm_prefill(int O, int I, int k, const void *planes_dev, const void *coeffs_dev, const uint16_t *X,
                      uint16_t *Y, int T, hipStream_t stream)
{
    int st = check_shape(O, I, k);
    if (st != SBVR_OK)
        return st;
    if (T < 1 || !planes_dev || !coeffs_dev || !X || !Y)
        return SBVR_E_INVALID_ARG;
    if (T > (1 << 22))  // keeps the token grid dimension below 2^16
        return SBVR_E_UNSUPPORTED;
    if (!aligned(planes_dev, 16) || !aligned(coeffs_dev, 16) || !aligned(X, 16) || !aligned(Y, 2))
        return SBVR_E_ALIGNMENT;
    return launch_prefill(make_dims(O, I, k), planes_dev, coeffs_dev, X, Y, T, stream);
}

int sbvr_decompress_indexed(int O, int I, int k, int n_sets, const void *planes_dev, const void *index_dev,
                            const void *table_dev, uint16_t *W, hipStream_t stream)
{
    int st = check_shape(O, I, k);
    if (st != SBVR_OK)
        return st;
    if ((st = check_sets(n_sets)) != SBVR_OK)
        return st;
    if (!planes_dev || !index_dev || !table_dev || !W)
        return SBVR_E_INVALID_ARG;
    if (!aligned(planes_dev, 16) || !aligned(index_dev, 16) || !aligned(table_dev, 16) || !aligned(W, 16))
        return SBVR_E_ALIGNMENT;
    return launch_decompress(make_dims(O, I, k), indexed_weights(planes_dev, index_dev, table_dev, n_sets), W,
                             stream);
}

}  // extern "C"
