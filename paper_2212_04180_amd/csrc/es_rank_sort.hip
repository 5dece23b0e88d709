// es_rank_sort.hip -- the sort behind the sort-based ranks: the composite
// keys of all runs (run, order key, member) in ascending order, by the
// rocPRIM radix sort (hipCUB interface), over only the bits they use.
#include <hipcub/hipcub.hpp>

#include "es_internal.hpp"

namespace esmi {

namespace {
int32_t bits_for(int64_t n)  // bits of the largest index n - 1 (0 for n = 1)
{
    int32_t b = 0;
    while (((int64_t)1 << b) < n) ++b;
    return b;
}
}  // namespace

void rank_sort_bits(const Geometry& g, int32_t* bn, int32_t* br)
{
    *bn = bits_for(g.N);
    *br = bits_for(g.R);
}

size_t rank_sort_temp_bytes(const Geometry& g)
{
    int32_t bn, br;
    rank_sort_bits(g, &bn, &br);
    size_t bytes = 0;
    const hipError_t e = hipcub::DeviceRadixSort::SortKeys(nullptr, bytes, (const uint64_t*)nullptr, (uint64_t*)nullptr,
                                                           (int)((int64_t)g.R * g.N), 0, 32 + bn + br, (hipStream_t)0);
    return e == hipSuccess ? (bytes ? bytes : 1) : 0;
}

hipError_t launch_rank_sort(const Geometry& g, const RankSortBuffers& rs, hipStream_t s)
{
    size_t bytes = rs.temp_bytes;
    return hipcub::DeviceRadixSort::SortKeys(rs.temp, bytes, (const uint64_t*)rs.kin, rs.kout, (int)((int64_t)g.R * g.N),
                                             0, 32 + rs.bn + rs.br, s);
}

}  // namespace esmi
