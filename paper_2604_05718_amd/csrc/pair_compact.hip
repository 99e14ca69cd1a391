// Mutual-pair test, RepMask and compact ids (Sec. 3.2, Alg. 1) for gfx950, the
// per-image cluster counts turned into offsets, and the reduction of the affinity
// kernel's partials to nearest neighbours.
//
// Compaction: one workgroup of 1024 threads per image. The neighbours of the
// image are gathered into LDS (reduced from the affinity kernel's per-tile
// partials, or read from nb). Each thread then takes a contiguous run of
// ceil(n/1024) tokens, counts the representatives in it (not in a mutual pair, or
// the lower index of one), and one workgroup-wide exclusive scan of the counts
// gives the id of the run's first representative, so ids follow the left-to-right
// scan of the paper. Partners then copy the id of their (lower-index)
// representative.
//
// Offsets: each image's workgroup stores its cluster count in y_off[b+1] as soon as
// its scan has it. With an arrival counter (the workspace's sync region), the
// workgroup whose arrival is counted last turns the counts into offsets in place
// once its own writes are issued, so the pair average reads each image's offset
// once instead of summing the counts before it; without one, a second
// one-workgroup launch does it. No workgroup ever waits for another.
#include "mpm_device.h"
#include "mpm_launch.h"

namespace mpm {
namespace {

constexpr int kCompactThreads = 1024;
constexpr int kCompactWaves = kCompactThreads / kWave;
constexpr int kPartialBatch = 8;  // partial tiles whose loads are issued together (16 spilled)
constexpr int kDoneSlot = 65535;  // sync-region slot of the images-done counter

__device__ __forceinline__ bool is_mutual(const int32_t* nbl, int i, int j, int n)
{
    return j >= 0 && j < n && j != i && nbl[j] == i;
}

// Exclusive prefix sum of one value per thread over the workgroup (wave scans
// by lane shuffles, wave totals through LDS); *total receives the sum.
__device__ __forceinline__ int block_exclusive_scan(int v, int32_t* wave_sum, int* total)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    int x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int y = __shfl_up(x, o);
        x += lane >= o ? y : 0;
    }
    if (lane == kWave - 1) wave_sum[wave] = x;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kCompactWaves; ++w) {
        const int c = wave_sum[w];
        before += w < wave ? c : 0;
        all += c;
    }
    *total = all;
    return before + x - v;
}

// Counts written by other workgroups of the same launch, which may run on another
// XCD whose L2 is not coherent with the writer's: agent-scope atomic stores and
// loads (sc1) are performed at the device's coherence point, so they need no cache
// write-back or invalidation. A writer waits until its stores have completed
// (vmcnt(0)) before it counts its arrival; the last one loads only after the
// counter told it every writer had arrived.
__device__ __forceinline__ void store_coherent(int32_t* p, int32_t v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int32_t load_coherent(const int32_t* p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// In-place offsets from counts: y_off[1..B] hold the cluster counts of the B images
// on entry and their inclusive prefix sums on exit; y_off[0] = 0.
template <bool COHERENT>
__device__ void scan_offsets(int32_t* y_off, int B, int32_t* wave_sum)
{
    const int tid = threadIdx.x;
    const int per = (B + kCompactThreads - 1) / kCompactThreads;
    const int k0 = min(B, tid * per);
    const int k1 = min(B, k0 + per);
    int s = 0;
    for (int k = k0; k < k1; ++k) s += COHERENT ? load_coherent(y_off + 1 + k) : y_off[1 + k];
    int total;
    int run = block_exclusive_scan(s, wave_sum, &total);
    // The sums go to the coherence point too, where the counts they replace were written.
    for (int k = k0; k < k1; ++k) {
        if (COHERENT) {
            run += load_coherent(y_off + 1 + k);
            store_coherent(y_off + 1 + k, run);
        } else {
            run += y_off[1 + k];
            y_off[1 + k] = run;
        }
    }
    if (tid == 0) {
        if (COHERENT) store_coherent(y_off, 0);
        else y_off[0] = 0;
    }
}

// FROM_PARTIALS: nb is first reduced from the affinity kernel's per-tile partials
// (larger score, then smaller index), written out, and kept in LDS; otherwise nb is
// read from memory into LDS. sync (may be null): arrival counters, zero on entry and
// on exit; with it the last workgroup scans the offsets.
template <bool FROM_PARTIALS>
__global__ __launch_bounds__(kCompactThreads) void pair_compact_kernel(
    const float* __restrict__ pv, const int32_t* __restrict__ pi, int T, int ct, int32_t* __restrict__ nb,
    const int32_t* __restrict__ x_off, int B, int N, int32_t* __restrict__ map, int32_t* __restrict__ src,
    int32_t* y_off, int32_t* sync)
{
    extern __shared__ int32_t lds[];
    int32_t* nbl = lds;       // nearest neighbour per token, N entries
    int32_t* rid = lds + N;   // compact id per representative, N entries
    __shared__ int32_t wave_sum[kCompactWaves];
    __shared__ int last;

    const int b = blockIdx.x;
    const int n = x_off ? x_off[b + 1] - x_off[b] : N;
    const int tid = threadIdx.x;

    if (FROM_PARTIALS) {
        const int tiles = (n + ct - 1) / ct;
        for (int i = tid; i < n; i += kCompactThreads) {
            float v = -__builtin_inff();
            int32_t j = -1;
            for (int t0 = 0; t0 < tiles; t0 += kPartialBatch) {
                float ov[kPartialBatch];
                int32_t oi[kPartialBatch];
#pragma unroll
                for (int u = 0; u < kPartialBatch; ++u) {
                    const long o = ((long)b * T + t0 + u) * N + i;
                    ov[u] = t0 + u < tiles ? pv[o] : -__builtin_inff();
                    oi[u] = t0 + u < tiles ? pi[o] : -1;
                }
#pragma unroll
                for (int u = 0; u < kPartialBatch; ++u) {
                    if (ov[u] > v || (ov[u] == v && (uint32_t)oi[u] < (uint32_t)j)) {
                        v = ov[u];
                        j = oi[u];
                    }
                }
            }
            nbl[i] = j;
            nb[(long)b * N + i] = j;
        }
    } else {
        for (int i = tid; i < n; i += kCompactThreads) nbl[i] = nb[(long)b * N + i];
    }
    __syncthreads();

    // This thread's run of tokens and the representatives in it.
    const int per = (n + kCompactThreads - 1) / kCompactThreads;
    const int i0 = min(n, tid * per);
    const int i1 = min(n, i0 + per);
    int reps = 0;
    for (int i = i0; i < i1; ++i) {
        const int j = nbl[i];
        reps += (!is_mutual(nbl, i, j, n) || i < j) ? 1 : 0;
    }
    int total;
    int id = block_exclusive_scan(reps, wave_sum, &total);
    // The image's count is final here: publish it and count the arrival now, so that the
    // atomic's round trip overlaps the src and map writes below (its result is read last).
    int arrived = 0;
    if (sync != nullptr && tid == 0) {
        store_coherent(y_off + b + 1, total);
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): the count is at the coherence point
        arrived = __hip_atomic_fetch_add(sync + kDoneSlot, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    for (int i = i0; i < i1; ++i) {
        const int j = nbl[i];
        const bool mutual = is_mutual(nbl, i, j, n);
        if (!mutual || i < j) {
            rid[i] = id;
            const long k = (long)b * N + id;
            src[2 * k] = i;
            src[2 * k + 1] = mutual ? j : i;
            ++id;
        }
    }
    __syncthreads();  // rid complete

    for (int i = tid; i < N; i += kCompactThreads) {
        int m = -1;
        if (i < n) {
            const int j = nbl[i];
            m = (is_mutual(nbl, i, j, n) && j < i) ? rid[j] : rid[i];
        }
        map[(long)b * N + i] = m;
    }
    if (sync == nullptr) {
        if (tid == 0) y_off[b + 1] = total;
        return;
    }
    if (tid == 0) last = arrived == B - 1;
    __syncthreads();
    if (!last) return;
    scan_offsets<true>(y_off, B, wave_sum);
    if (tid == 0) store_coherent(sync + kDoneSlot, 0);
}

__global__ __launch_bounds__(kCompactThreads) void offsets_kernel(int32_t* y_off, int B)
{
    __shared__ int32_t wave_sum[kCompactWaves];
    scan_offsets<false>(y_off, B, wave_sum);
}

// Sum of squares of one 16-byte group of storage values, in float32.
__device__ __forceinline__ float sumsq16(u32x4 a, float s, Bf16)
{
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        s = fmaf(bf16_lo(a[e]), bf16_lo(a[e]), s);
        s = fmaf(bf16_hi(a[e]), bf16_hi(a[e]), s);
    }
    return s;
}

__device__ __forceinline__ float sumsq16(u32x4 a, float s, F32)
{
#pragma unroll
    for (int e = 0; e < 4; ++e) s = fmaf(__uint_as_float(a[e]), __uint_as_float(a[e]), s);
    return s;
}

// nb[b*N + i] = lexicographic max over the candidate-tile partials of row i
// (larger score, then smaller index); optional cosine of the chosen pair.
template <class S>
__global__ __launch_bounds__(256) void reduce_partials_kernel(const float* __restrict__ pv,
                                                               const int32_t* __restrict__ pi,
                                                               const uint8_t* __restrict__ x,
                                                               const int32_t* __restrict__ x_off, int B, int N,
                                                               int D, int T, int ct, int32_t* __restrict__ nb,
                                                               float* __restrict__ best)
{
    const long g = (long)blockIdx.x * 256 + threadIdx.x;
    if (g >= (long)B * N) return;
    const int b = (int)(g / N);
    const int i = (int)(g - (long)b * N);
    const int row0 = x_off ? x_off[b] : b * N;
    const int n = x_off ? x_off[b + 1] - row0 : N;
    if (i >= n) return;
    const int tiles = (n + ct - 1) / ct;
    float v = -__builtin_inff();
    int32_t j = -1;
    // The partials of 8 tiles are loaded before any is merged, so their loads overlap.
    constexpr int kBatch = 8;
    for (int t0 = 0; t0 < tiles; t0 += kBatch) {
        float ov[kBatch];
        int32_t oi[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const long o = ((long)b * T + t0 + u) * N + i;
            ov[u] = t0 + u < tiles ? pv[o] : -__builtin_inff();
            oi[u] = t0 + u < tiles ? pi[o] : -1;
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            if (ov[u] > v || (ov[u] == v && (uint32_t)oi[u] < (uint32_t)j)) {
                v = ov[u];
                j = oi[u];
            }
        }
    }
    nb[g] = j;
    if (best) {
        // Diagnostic only: divide by the query's own norm to report the cosine.
        const long rowbytes = (long)D * S::kBytes;
        const uint8_t* xr = x + ((long)row0 + i) * rowbytes;
        float t2 = 0.0f;
        for (long kk = 0; kk < rowbytes; kk += 16) t2 = sumsq16(load16(xr + kk), t2, S{});
        best[g] = j >= 0 ? v / fmaxf(sqrtf(t2), 1e-12f) : -__builtin_inff();
    }
}

// Zeroes `words` 32-bit words (the workspace's sync region) with plain stores.
__global__ __launch_bounds__(256) void zero_words_kernel(int32_t* p, long words)
{
    for (long k = (long)blockIdx.x * 256 + threadIdx.x; k < words; k += (long)gridDim.x * 256) p[k] = 0;
}

template <bool FROM_PARTIALS>
hipError_t launch_compact_t(const float* pv, const int32_t* pi, int T, int ct, int32_t* nb, const int32_t* x_off,
                            int B, int N, int32_t* map, int32_t* src, int32_t* y_off, int32_t* sync,
                            hipStream_t stream)
{
    const size_t lds = 2 * (size_t)N * sizeof(int32_t);
    if (lds > 32768) {
        const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(pair_compact_kernel<FROM_PARTIALS>),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(pair_compact_kernel<FROM_PARTIALS>, dim3(B), dim3(kCompactThreads), lds, stream, pv, pi, T, ct,
                       nb, x_off, B, N, map, src, y_off, sync);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || sync != nullptr) return e;
    hipLaunchKernelGGL(offsets_kernel, dim3(1), dim3(kCompactThreads), 0, stream, y_off, B);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_pair_compact(const int32_t* nb, const int32_t* x_off, int B, int N, int32_t* map, int32_t* src,
                               int32_t* y_off, int32_t* sync, hipStream_t stream)
{
    return launch_compact_t<false>(nullptr, nullptr, 0, 1, const_cast<int32_t*>(nb), x_off, B, N, map, src, y_off,
                                   sync, stream);
}

hipError_t launch_pair_compact_partials(const float* pv, const int32_t* pi, int T, int ct, int32_t* nb,
                                        const int32_t* x_off, int B, int N, int32_t* map, int32_t* src,
                                        int32_t* y_off, int32_t* sync, hipStream_t stream)
{
    return launch_compact_t<true>(pv, pi, T, ct, nb, x_off, B, N, map, src, y_off, sync, stream);
}

hipError_t launch_reduce_partials(const float* pv, const int32_t* pi, int ct, const void* x, const int32_t* x_off,
                                  int B, int N, int D, int dt, int32_t* nb, float* best, hipStream_t stream)
{
    const int T = partial_tiles(N);
    const long total = (long)B * N;
    const dim3 grid((unsigned)((total + 255) / 256));
    const uint8_t* xp = static_cast<const uint8_t*>(x);
    if (dt == kBf16)
        hipLaunchKernelGGL(reduce_partials_kernel<Bf16>, grid, dim3(256), 0, stream, pv, pi, xp, x_off, B, N, D, T, ct,
                           nb, best);
    else
        hipLaunchKernelGGL(reduce_partials_kernel<F32>, grid, dim3(256), 0, stream, pv, pi, xp, x_off, B, N, D, T, ct,
                           nb, best);
    return hipGetLastError();
}

hipError_t launch_zero_words(int32_t* p, long words, hipStream_t stream)
{
    const long blocks = (words + 255) / 256;
    hipLaunchKernelGGL(zero_words_kernel, dim3((unsigned)(blocks < 1024 ? blocks : 1024)), dim3(256), 0, stream, p,
                       words);
    return hipGetLastError();
}

}  // namespace mpm
