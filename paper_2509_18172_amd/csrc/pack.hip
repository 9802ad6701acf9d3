// Repacking between the canonical SBVR tensors and the device format
// (layout.h), one thread per 32-bit plane word / coefficient.  Every byte of
// the device buffers is written (padding with zeros), so they need no prior
// clearing.
#include "launch.h"

namespace sbvr {

__global__ void pack_planes_kernel(Dims d, const uint32_t *__restrict__ canon,
                                   uint32_t *__restrict__ dev, size_t total)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    const size_t bw = plane_block_words(d.k);
    const size_t blk = idx / bw;
    const int within = (int)(idx % bw);
    const int slot = within / 4, w = within % 4;
    const int i = slot % d.k, br = slot / d.k;
    const int r = br % d.tr, b = br / d.tr;
    const int o = (int)(blk / d.n_gblocks) * d.tr + r;
    const int g = (int)(blk % d.n_gblocks) * GB + b;
    uint32_t v = 0;
    if (o < d.O && g < d.G)
        v = to_device_word(canon[(((size_t)o * d.G + g) * d.k + i) * 4 + w]);
    dev[idx] = v;
}

__global__ void unpack_planes_kernel(Dims d, const uint32_t *__restrict__ dev,
                                     uint32_t *__restrict__ canon, size_t total)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    const int w = (int)(idx % 4);
    const size_t rest = idx / 4;
    const int i = (int)(rest % d.k);
    const size_t og = rest / d.k;
    const int g = (int)(og % d.G), o = (int)(og / d.G);
    const size_t blk = (size_t)(o / d.tr) * d.n_gblocks + g / GB;
    const int slot = ((g % GB) * d.tr + o % d.tr) * d.k + i;
    canon[idx] = to_canonical_word(dev[blk * plane_block_words(d.k) + slot * 4 + w]);
}

__global__ void pack_coeffs_kernel(Dims d, const uint16_t *__restrict__ canon,
                                   uint16_t *__restrict__ dev, size_t total)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    const size_t be = coeff_block_entries(d.k);
    const size_t blk = idx / be;
    const int within = (int)(idx % be);
    // entry (q * GB + b) * CPL + j holds A row m = 4q + j = (r, i) of slot b
    const int cpl = coefs_per_quad(d.k), rs = row_slots(d.k);
    const int j = within % cpl, b = (within / cpl) % GB, q = within / (cpl * GB);
    const int m = 4 * q + j;
    const int r = m / rs, i = m % rs;
    const int o = (int)(blk / d.n_gblocks) * d.tr + r;
    const int g = (int)(blk % d.n_gblocks) * GB + b;
    uint16_t v = 0;
    if (o < d.O && g < d.G)
        v = canon[((size_t)o * d.G + g) * d.k + i];
    dev[idx] = v;
}

__global__ void unpack_coeffs_kernel(Dims d, const uint16_t *__restrict__ dev,
                                     uint16_t *__restrict__ canon, size_t total)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    const int i = (int)(idx % d.k);
    const size_t og = idx / d.k;
    const int g = (int)(og % d.G), o = (int)(og / d.G);
    const size_t blk = (size_t)(o / d.tr) * d.n_gblocks + g / GB;
    canon[idx] = dev[blk * coeff_block_entries(d.k) + coeff_entry(d.k, o % d.tr, g % GB, i)];
}

// Coefficient-cache format (Sec. 4.4): index blocks (layout.h) and the table
// of coefficient sets, TABLE_STRIDE entries per set.
__global__ void pack_index_kernel(Dims d, const uint16_t *__restrict__ canon,
                                  uint16_t *__restrict__ dev, size_t total)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    const size_t be = index_block_entries(d.k);
    const size_t blk = idx / be;
    const int e = (int)(idx % be);
    // entry ((r / NP) * GB + b) * NP + r % NP
    const int np = index_per_lane(d.k);
    const int p = e % np, b = (e / np) % GB, q = e / (np * GB);
    const int o = (int)(blk / d.n_gblocks) * d.tr + q * np + p;
    const int g = (int)(blk % d.n_gblocks) * GB + b;
    dev[idx] = (o < d.O && g < d.G) ? canon[(size_t)o * d.G + g] : (uint16_t)0;
}

__global__ void unpack_index_kernel(Dims d, const uint16_t *__restrict__ dev,
                                    uint16_t *__restrict__ canon, size_t total)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    const int g = (int)(idx % d.G), o = (int)(idx / d.G);
    const size_t blk = (size_t)(o / d.tr) * d.n_gblocks + g / GB;
    canon[idx] = dev[blk * index_block_entries(d.k) + index_entry(d.k, o % d.tr, g % GB)];
}

__global__ void pack_table_kernel(int k, const uint16_t *__restrict__ canon, uint16_t *__restrict__ dev,
                                  size_t total)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    const size_t n = idx / TABLE_STRIDE;
    const int i = (int)(idx % TABLE_STRIDE);
    dev[idx] = i < k ? canon[n * k + i] : (uint16_t)0;
}

__global__ void unpack_table_kernel(int k, const uint16_t *__restrict__ dev, uint16_t *__restrict__ canon,
                                    size_t total)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    canon[idx] = dev[(idx / k) * TABLE_STRIDE + idx % k];
}

static unsigned grid_for(size_t total) { return (unsigned)((total + 255) / 256); }

int launch_pack(const Dims &d0, const uint32_t *planes_canon, const uint16_t *coeffs_canon,
                void *planes_dev, void *coeffs_dev, hipStream_t stream)
{
    Dims d = d0;
    size_t pw = plane_bytes(d) / 4, ce = coeff_bytes(d) / 2;
    uint32_t *pd = (uint32_t *)planes_dev;
    uint16_t *cd = (uint16_t *)coeffs_dev;
    void *pargs[] = {&d, &planes_canon, &pd, &pw};
    int st = launch_kernel((const void *)pack_planes_kernel, dim3(grid_for(pw)), dim3(256), 0, stream, pargs);
    if (st != SBVR_OK)
        return st;
    void *cargs[] = {&d, &coeffs_canon, &cd, &ce};
    return launch_kernel((const void *)pack_coeffs_kernel, dim3(grid_for(ce)), dim3(256), 0, stream, cargs);
}

int launch_unpack(const Dims &d0, const void *planes_dev, const void *coeffs_dev,
                  uint32_t *planes_canon, uint16_t *coeffs_canon, hipStream_t stream)
{
    Dims d = d0;
    size_t pw = (size_t)d.O * d.G * d.k * 4, ce = (size_t)d.O * d.G * d.k;
    const uint32_t *pd = (const uint32_t *)planes_dev;
    const uint16_t *cd = (const uint16_t *)coeffs_dev;
    void *pargs[] = {&d, &pd, &planes_canon, &pw};
    int st = launch_kernel((const void *)unpack_planes_kernel, dim3(grid_for(pw)), dim3(256), 0, stream, pargs);
    if (st != SBVR_OK)
        return st;
    void *cargs[] = {&d, &cd, &coeffs_canon, &ce};
    return launch_kernel((const void *)unpack_coeffs_kernel, dim3(grid_for(ce)), dim3(256), 0, stream, cargs);
}

int launch_pack_indexed(const Dims &d0, int n_sets, const uint32_t *planes_canon, const uint16_t *index_canon,
                        const uint16_t *table_canon, void *planes_dev, void *index_dev, void *table_dev,
                        hipStream_t stream)
{
    Dims d = d0;
    int k = d.k;
    size_t pw = plane_bytes(d) / 4, ie = index_bytes(d) / 2, te = (size_t)n_sets * TABLE_STRIDE;
    uint32_t *pd = (uint32_t *)planes_dev;
    uint16_t *id = (uint16_t *)index_dev, *td = (uint16_t *)table_dev;
    void *pargs[] = {&d, &planes_canon, &pd, &pw};
    int st = launch_kernel((const void *)pack_planes_kernel, dim3(grid_for(pw)), dim3(256), 0, stream, pargs);
    if (st != SBVR_OK)
        return st;
    void *iargs[] = {&d, &index_canon, &id, &ie};
    st = launch_kernel((const void *)pack_index_kernel, dim3(grid_for(ie)), dim3(256), 0, stream, iargs);
    if (st != SBVR_OK)
        return st;
    void *targs[] = {&k, &table_canon, &td, &te};
    return launch_kernel((const void *)pack_table_kernel, dim3(grid_for(te)), dim3(256), 0, stream, targs);
}

int launch_unpack_indexed(const Dims &d0, int n_sets, const void *planes_dev, const void *index_dev,
                          const void *table_dev, uint32_t *planes_canon, uint16_t *index_canon,
                          uint16_t *table_canon, hipStream_t stream)
{
    Dims d = d0;
    int k = d.k;
    size_t pw = (size_t)d.O * d.G * d.k * 4, ie = (size_t)d.O * d.G, te = (size_t)n_sets * d.k;
    const uint32_t *pd = (const uint32_t *)planes_dev;
    const uint16_t *id = (const uint16_t *)index_dev, *td = (const uint16_t *)table_dev;
    void *pargs[] = {&d, &pd, &planes_canon, &pw};
    int st = launch_kernel((const void *)unpack_planes_kernel, dim3(grid_for(pw)), dim3(256), 0, stream, pargs);
    if (st != SBVR_OK)
        return st;
    void *iargs[] = {&d, &id, &index_canon, &ie};
    st = launch_kernel((const void *)unpack_index_kernel, dim3(grid_for(ie)), dim3(256), 0, stream, iargs);
    if (st != SBVR_OK)
        return st;
    void *targs[] = {&k, &td, &table_canon, &te};
    return launch_kernel((const void *)unpack_table_kernel, dim3(grid_for(te)), dim3(256), 0, stream, targs);
}

}  // namespace sbvr
