// Mutual-pair test, RepMask and compact ids (Sec. 3.2, Alg. 1) for gfx950.
//
// One workgroup of 1024 threads per image. Tokens are visited in rounds of
// 1024; in each round every thread decides whether its token is a
// representative (not in a mutual pair, or the lower index of one), the wave
// ballots the flags and each lane's rank inside the wave is the popcount of
// the ballot below it; wave totals are scanned through LDS. A running base
// carries the count across rounds, so ids follow the left-to-right scan of
// the paper. Neighbours and representative ids are kept in LDS, and partners
// then copy the id of their (lower-index) representative.
#include "mpm_device.h"
#include "mpm_launch.h"

namespace mpm {
namespace {

constexpr int kCompactThreads = 1024;
constexpr int kCompactWaves = kCompactThreads / kWave;

__device__ __forceinline__ bool is_mutual(const int32_t* nbl, int i, int j, int n)
{
    return j >= 0 && j < n && j != i && nbl[j] == i;
}

// FROM_PARTIALS: nb is first reduced from the affinity kernel's per-tile
// partials (larger score, then smaller index), written out, and kept in LDS;
// otherwise nb is read from memory into LDS.
template <bool FROM_PARTIALS>
__global__ __launch_bounds__(kCompactThreads) void pair_compact_kernel(
    const float* __restrict__ pv, const int32_t* __restrict__ pi, int T, int ct, int32_t* __restrict__ nb,
    const int32_t* __restrict__ x_off, int N, int32_t* __restrict__ map, int32_t* __restrict__ src,
    int32_t* __restrict__ count)
{
    extern __shared__ int32_t lds[];
    int32_t* nbl = lds;       // nearest neighbour per token, N entries
    int32_t* rid = lds + N;   // compact id per representative, N entries
    __shared__ int32_t wave_total[kCompactWaves];

    const int b = blockIdx.x;
    const int n = x_off ? x_off[b + 1] - x_off[b] : N;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));

    if (FROM_PARTIALS) {
        const int tiles = (n + ct - 1) / ct;
        for (int i = tid; i < n; i += kCompactThreads) {
            float v = -__builtin_inff();
            int32_t j = -1;
            for (int t = 0; t < tiles; ++t) {
                const long o = ((long)b * T + t) * N + i;
                const float ov = pv[o];
                const int32_t oi = pi[o];
                if (ov > v || (ov == v && (uint32_t)oi < (uint32_t)j)) {
                    v = ov;
                    j = oi;
                }
            }
            nbl[i] = j;
            nb[(long)b * N + i] = j;
        }
    } else {
        for (int i = tid; i < n; i += kCompactThreads) nbl[i] = nb[(long)b * N + i];
    }
    __syncthreads();

    int base = 0;
    for (int i0 = 0; i0 < n; i0 += kCompactThreads) {
        const int i = i0 + tid;
        int j = -1;
        bool mutual = false, rep = false;
        if (i < n) {
            j = nbl[i];
            mutual = is_mutual(nbl, i, j, n);
            rep = !mutual || i < j;
        }
        const uint64_t ballot = __ballot(rep);
        const int rank = __popcll(ballot & below);
        if (lane == 0) wave_total[wave] = __popcll(ballot);
        __syncthreads();
        int before = 0, round_total = 0;
#pragma unroll
        for (int w = 0; w < kCompactWaves; ++w) {
            const int c = wave_total[w];
            before += (w < wave) ? c : 0;
            round_total += c;
        }
        if (rep) {
            const int id = base + before + rank;
            rid[i] = id;
            const long k = (long)b * N + id;
            src[2 * k] = i;
            src[2 * k + 1] = mutual ? j : i;
        }
        base += round_total;
        __syncthreads();  // wave_total is rewritten next round; rid complete after the last
    }

    for (int i = tid; i < N; i += kCompactThreads) {
        int id = -1;
        if (i < n) {
            const int j = nbl[i];
            id = (is_mutual(nbl, i, j, n) && j < i) ? rid[j] : rid[i];
        }
        map[(long)b * N + i] = id;
    }
    if (tid == 0) count[b] = base;
}

template <bool FROM_PARTIALS>
hipError_t launch_compact_t(const float* pv, const int32_t* pi, int T, int ct, int32_t* nb, const int32_t* x_off,
                            int B, int N, int32_t* map, int32_t* src, int32_t* count, hipStream_t stream)
{
    const size_t lds = 2 * (size_t)N * sizeof(int32_t);
    if (lds > 32768) {
        const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(pair_compact_kernel<FROM_PARTIALS>),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(pair_compact_kernel<FROM_PARTIALS>, dim3(B), dim3(kCompactThreads), lds, stream, pv, pi, T, ct,
                       nb, x_off, N, map, src, count);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_pair_compact(const int32_t* nb, const int32_t* x_off, int B, int N, int32_t* map, int32_t* src,
                               int32_t* count, hipStream_t stream)
{
    return launch_compact_t<false>(nullptr, nullptr, 0, 1, const_cast<int32_t*>(nb), x_off, B, N, map, src, count,
                                   stream);
}

hipError_t launch_pair_compact_partials(const float* pv, const int32_t* pi, int T, int ct, int32_t* nb,
                                        const int32_t* x_off, int B, int N, int32_t* map, int32_t* src,
                                        int32_t* count, hipStream_t stream)
{
    return launch_compact_t<true>(pv, pi, T, ct, nb, x_off, B, N, map, src, count, stream);
}

}  // namespace mpm
