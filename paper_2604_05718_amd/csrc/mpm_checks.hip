// Device-side validation of the data-dependent preconditions of the C ABI (the
// library's checked mode). Each kernel reads caller data that the operation itself
// would index with, and ORs a violation bit into one device word; it never writes
// anything else. Every read is bounded by the shape alone (B, N, D and the counts,
// clamped to [0, N]), so garbage offsets or values cannot take a check out of bounds.
// Offsets are checked (and the verdict read back) before any check that walks rows
// through them.
#include "mpm_device.h"
#include "mpm_launch.h"

namespace mpm {
namespace {

constexpr int kCheckThreads = 256;

__device__ __forceinline__ void report(int32_t* verdict, int32_t bit)
{
    __hip_atomic_fetch_or(verdict, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Tokens of image b under optional packed offsets, clamped to [0, N].
__device__ __forceinline__ int count_of(const int32_t* off, int b, int N)
{
    if (off == nullptr) return N;
    return min(max(off[b + 1] - off[b], 0), N);
}

// Packed offsets: off[0] >= 0, lo_n <= off[b+1] - off[b] <= N (so non-decreasing),
// off[B] <= cap when cap >= 0, and, with `within` (the counts of the images the rows
// come from), at most that many rows per image.
__global__ __launch_bounds__(kCheckThreads) void check_offsets_kernel(const int32_t* off, int B, int N, int lo_n,
                                                                      long cap, const int32_t* within,
                                                                      int32_t* verdict)
{
    const int b = blockIdx.x * kCheckThreads + threadIdx.x;
    if (b >= B) return;
    const int o0 = off[b], o1 = off[b + 1];
    const long n = (long)o1 - (long)o0;
    bool bad = o0 < 0 || n < lo_n || n > N || (b == B - 1 && cap >= 0 && o1 > cap);
    if (!bad && within != nullptr) bad = n > count_of(within, b, N);
    if (bad) report(verdict, kCheckOffsets);
}

// Slot values v[b*N + i] (`per` values per slot, consecutive) for i < count_of(cnt_off, b):
// each in [lo, hi_b), hi_b = count_of(hi_off, b, N) (hi_off null: N).
__global__ __launch_bounds__(kCheckThreads) void check_slots_kernel(const int32_t* v, int per, const int32_t* cnt_off,
                                                                    int lo, const int32_t* hi_off, int B, int N,
                                                                    int32_t bit, int32_t* verdict)
{
    const int b = blockIdx.y;
    const int i = blockIdx.x * kCheckThreads + threadIdx.x;
    if (i >= count_of(cnt_off, b, N)) return;
    const int hi = count_of(hi_off, b, N);
    bool bad = false;
    for (int e = 0; e < per; ++e) {
        const int x = v[((long)b * N + i) * per + e];
        bad |= x < lo || x >= hi;
    }
    if (bad) report(verdict, bit);
}

// Neighbours as the compaction reads them: nb[i] in [0, n_b) and not i, or -1 when n_b == 1.
__global__ __launch_bounds__(kCheckThreads) void check_nb_kernel(const int32_t* nb, const int32_t* x_off, int B, int N,
                                                                 int32_t* verdict)
{
    const int b = blockIdx.y;
    const int i = blockIdx.x * kCheckThreads + threadIdx.x;
    const int n = count_of(x_off, b, N);
    if (i >= n) return;
    const int j = nb[(long)b * N + i];
    const bool ok = n == 1 ? j == -1 : (j >= 0 && j < n && j != i);
    if (!ok) report(verdict, kCheckValues);
}

// Grid positions of a locality-constrained insertion: in [0, limit) and non-decreasing in
// grid row along each image.
__global__ __launch_bounds__(kCheckThreads) void check_pos_kernel(const int32_t* pos, const int32_t* x_off, int B,
                                                                  int N, int grid_w, long limit, int32_t* verdict)
{
    const int b = blockIdx.y;
    const int i = blockIdx.x * kCheckThreads + threadIdx.x;
    const int n = count_of(x_off, b, N);
    if (i >= n) return;
    const long row0 = x_off ? x_off[b] : (long)b * N;
    const int p = pos[row0 + i];
    bool bad = p < 0 || (long)p >= limit;
    if (!bad && i > 0) {
        const int q = pos[row0 + i - 1];
        bad = q >= 0 && q / grid_w > p / grid_w;
    }
    if (bad) report(verdict, kCheckPositions);
}

// Given inverse norms: finite and positive, one per token.
__global__ __launch_bounds__(kCheckThreads) void check_inv_kernel(const float* inv, const int32_t* x_off, int B, int N,
                                                                  int32_t* verdict)
{
    const int b = blockIdx.y;
    const int i = blockIdx.x * kCheckThreads + threadIdx.x;
    if (i >= count_of(x_off, b, N)) return;
    const float v = inv[(x_off ? (long)x_off[b] : (long)b * N) + i];
    if (!(v > 0.0f && v < __builtin_inff())) report(verdict, kCheckValues);
}

// Token values finite (16-byte vectors, grid-stride over each image's rows).
template <class S>
__global__ __launch_bounds__(kCheckThreads) void check_finite_kernel(const uint8_t* x, const int32_t* x_off, int B,
                                                                     int N, int D, int32_t* verdict)
{
    const int b = blockIdx.y;
    const int n = count_of(x_off, b, N);
    const long vpr = (long)D * S::kBytes / 16;
    const long total = (long)n * vpr;
    const uint8_t* img = x + (x_off ? (long)x_off[b] : (long)b * N) * vpr * 16;
    bool bad = false;
    for (long f = (long)blockIdx.x * kCheckThreads + threadIdx.x; f < total; f += (long)gridDim.x * kCheckThreads) {
        const u32x4 v = load16(img + f * 16);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t w = v[e];
            if (S::kBytes == 2) bad |= (w & 0x7f80u) == 0x7f80u || (w & 0x7f800000u) == 0x7f800000u;
            else bad |= (w & 0x7f800000u) == 0x7f800000u;
        }
    }
    if (bad) report(verdict, kCheckValues);
}

dim3 slot_grid(int B, int N) { return dim3((unsigned)((N + kCheckThreads - 1) / kCheckThreads), (unsigned)B); }

}  // namespace

hipError_t launch_check_offsets(const int32_t* off, int B, int N, int lo_n, long cap, const int32_t* within,
                                int32_t* verdict, hipStream_t stream)
{
    hipLaunchKernelGGL(check_offsets_kernel, dim3((unsigned)((B + kCheckThreads - 1) / kCheckThreads)),
                       dim3(kCheckThreads), 0, stream, off, B, N, lo_n, cap, within, verdict);
    return hipGetLastError();
}

hipError_t launch_check_slots(const int32_t* v, int per, const int32_t* cnt_off, int lo, const int32_t* hi_off, int B,
                              int N, int32_t bit, int32_t* verdict, hipStream_t stream)
{
    hipLaunchKernelGGL(check_slots_kernel, slot_grid(B, N), dim3(kCheckThreads), 0, stream, v, per, cnt_off, lo, hi_off,
                       B, N, bit, verdict);
    return hipGetLastError();
}

hipError_t launch_check_nb(const int32_t* nb, const int32_t* x_off, int B, int N, int32_t* verdict, hipStream_t stream)
{
    hipLaunchKernelGGL(check_nb_kernel, slot_grid(B, N), dim3(kCheckThreads), 0, stream, nb, x_off, B, N, verdict);
    return hipGetLastError();
}

hipError_t launch_check_pos(const int32_t* pos, const int32_t* x_off, int B, int N, int grid_w, long limit,
                            int32_t* verdict, hipStream_t stream)
{
    hipLaunchKernelGGL(check_pos_kernel, slot_grid(B, N), dim3(kCheckThreads), 0, stream, pos, x_off, B, N, grid_w,
                       limit, verdict);
    return hipGetLastError();
}

hipError_t launch_check_inv(const float* inv, const int32_t* x_off, int B, int N, int32_t* verdict,
                            hipStream_t stream)
{
    hipLaunchKernelGGL(check_inv_kernel, slot_grid(B, N), dim3(kCheckThreads), 0, stream, inv, x_off, B, N, verdict);
    return hipGetLastError();
}

hipError_t launch_check_finite(const void* x, const int32_t* x_off, int B, int N, int D, int dt, int32_t* verdict,
                               hipStream_t stream)
{
    const dim3 grid(8, (unsigned)B);
    const uint8_t* xp = static_cast<const uint8_t*>(x);
    if (dt == kBf16)
        hipLaunchKernelGGL(check_finite_kernel<Bf16>, grid, dim3(kCheckThreads), 0, stream, xp, x_off, B, N, D, verdict);
    else
        hipLaunchKernelGGL(check_finite_kernel<F32>, grid, dim3(kCheckThreads), 0, stream, xp, x_off, B, N, D, verdict);
    return hipGetLastError();
}

}  // namespace mpm
