// es_rank_sort.hip -- the sort behind the sort-based ranks: every run's
// composite keys (order key << 32 | member) in ascending order, by the
// rocPRIM radix sort (hipCUB interface).  One run: the device-wide sort;
// several: the segmented sort over the runs' slices [r N, (r + 1) N).
#include <hipcub/hipcub.hpp>

#include "es_internal.hpp"

namespace esmi {

size_t rank_sort_temp_bytes(const Geometry& g)
{
    const int64_t total = (int64_t)g.R * g.N;
    size_t bytes = 0;
    hipError_t e;
    if (g.R == 1)
        e = hipcub::DeviceRadixSort::SortKeys(nullptr, bytes, (const uint64_t*)nullptr, (uint64_t*)nullptr,
                                              (int)total, 0, 64, (hipStream_t)0);
    else
        e = hipcub::DeviceSegmentedRadixSort::SortKeys(nullptr, bytes, (const uint64_t*)nullptr, (uint64_t*)nullptr,
                                                       (int)total, g.R, (const int32_t*)nullptr,
                                                       (const int32_t*)nullptr, 0, 64, (hipStream_t)0);
    return e == hipSuccess ? (bytes ? bytes : 1) : 0;
}

hipError_t launch_rank_sort(const Geometry& g, const RankSortBuffers& rs, hipStream_t s)
{
    const int64_t total = (int64_t)g.R * g.N;
    size_t bytes = rs.temp_bytes;
    if (g.R == 1)
        return hipcub::DeviceRadixSort::SortKeys(rs.temp, bytes, (const uint64_t*)rs.kin, rs.kout, (int)total, 0, 64, s);
    return hipcub::DeviceSegmentedRadixSort::SortKeys(rs.temp, bytes, (const uint64_t*)rs.kin, rs.kout, (int)total, g.R,
                                                      (const int32_t*)rs.offsets, (const int32_t*)rs.offsets + 1, 0,
                                                      64, s);
}

}  // namespace esmi
