/*
 * Drives the host side of the C ABI (include/mpm.h) for a build of the library's
 * host code with AddressSanitizer and UndefinedBehaviorSanitizer: every argument
 * check, the workspace layout arithmetic at the largest shapes, and, when run with
 * MPM_FAULT_INJECT=launch, the injected launch failure of every launching entry
 * point. No call here reaches a kernel launch, so no GPU is needed. Exits 0 when
 * every call returned the status its contract states.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../include/mpm.h"

#define EXPECT(call, want)                                                              \
    do {                                                                                \
        const int got_ = (call);                                                        \
        if (got_ != (want)) {                                                           \
            fprintf(stderr, "line %d: %s returned %d, expected %d\n", __LINE__, #call, got_, (int)(want)); \
            return 1;                                                                   \
        }                                                                               \
    } while (0)

int main(void)
{
    const int inject = getenv("MPM_FAULT_INJECT") != NULL && strcmp(getenv("MPM_FAULT_INJECT"), "launch") == 0;
    /* Stand-in device pointers: aligned, never dereferenced on the host. */
    void* A = (void*)(uintptr_t)0x100000;
    void* A2 = (void*)(uintptr_t)0x200000;
    void* MIS = (void*)(uintptr_t)0x100004;
    const size_t big = (size_t)1 << 40;

    /* Workspace arithmetic at the largest shapes the ABI accepts. */
    for (int32_t B = 1; B <= MPM_MAX_B; B = B * 3 + 1)
        for (int32_t N = 1; N <= MPM_MAX_N; N = N * 5 + 3) {
            const size_t w = mpm_workspace_bytes(B, N);
            size_t o[5];
            EXPECT(mpm_workspace_offsets(B, N, &o[0], &o[1], &o[2], &o[3], &o[4]), MPM_OK);
            if (!(o[0] == 0 && o[0] < o[1] && o[1] < o[2] && o[2] < o[3] && o[3] < o[4] && o[4] < w)) {
                fprintf(stderr, "workspace layout out of order at B=%d N=%d\n", B, N);
                return 1;
            }
        }
    EXPECT((int)mpm_workspace_bytes(0, 1), 0);
    EXPECT(mpm_workspace_offsets(1, 0, NULL, NULL, NULL, NULL, NULL), MPM_ERR_INVALID_ARG);

    /* Argument checks (no launch). */
    EXPECT(mpm_affinity(A, NULL, NULL, 0, 16, 64, MPM_BF16, 0, A, big, NULL, NULL, NULL), MPM_ERR_INVALID_ARG);
    EXPECT(mpm_affinity(A, NULL, NULL, 2, 16, 12, MPM_BF16, 0, A, big, NULL, NULL, NULL), MPM_ERR_INVALID_ARG);
    EXPECT(mpm_affinity(A, NULL, NULL, 2, 16, 64, MPM_BF16, 7, A, big, NULL, NULL, NULL), MPM_ERR_INVALID_ARG);
    EXPECT(mpm_affinity(MIS, NULL, NULL, 2, 16, 64, MPM_BF16, 0, A, big, NULL, NULL, NULL), MPM_ERR_INVALID_ARG);
    EXPECT(mpm_affinity(A, NULL, NULL, 2, MPM_MAX_N + 1, 64, MPM_BF16, 0, A, big, NULL, NULL, NULL),
           MPM_ERR_UNSUPPORTED);
    EXPECT(mpm_affinity(A, NULL, A, 2, 16, 64, MPM_F32, 0, A, big, NULL, NULL, NULL), MPM_ERR_UNSUPPORTED);
    EXPECT(mpm_affinity(A, NULL, NULL, 2, 16, 64, MPM_BF16, 0, A, 16, NULL, NULL, NULL), MPM_ERR_WORKSPACE);
    EXPECT(mpm_merge(A, NULL, NULL, 2, 16, 64, MPM_BF16, 0, NULL, A2, NULL, A2, A, big, NULL), MPM_ERR_INVALID_ARG);
    EXPECT(mpm_merge_noalloc(A, NULL, NULL, 64, 4096, 64, MPM_BF16, 0, A2, A2, NULL, A2, NULL), MPM_ERR_WORKSPACE);
    EXPECT(mpm_pair_compact(A, NULL, 2, 8, A, A, NULL, NULL), MPM_ERR_INVALID_ARG);
    EXPECT(mpm_pair_average(A, NULL, A, A, 2, 8, 64, MPM_BF16, MIS, NULL, NULL), MPM_ERR_INVALID_ARG);
    EXPECT(mpm_compose(A, NULL, 2, 8, A, NULL), MPM_ERR_INVALID_ARG);
    EXPECT(mpm_unmerge(A, NULL, A, NULL, -1, 2, 8, 64, MPM_BF16, A, NULL), MPM_ERR_INVALID_ARG);
    EXPECT(mpm_compose_unmerge(A, NULL, A, A2, A, NULL, 0, 2, 8, 64, MPM_BF16, A, NULL), MPM_ERR_INVALID_ARG);
    EXPECT(mpm_workspace_init(MIS, big, NULL), MPM_ERR_INVALID_ARG);
    EXPECT(mpm_merge_local(A, NULL, NULL, NULL, 2, 64, 64, MPM_BF16, 0, 1, 0, A2, A2, NULL, A2, A2, A, big, NULL, NULL,
                           NULL), MPM_ERR_INVALID_ARG);                                 /* grid_w < 1 */
    EXPECT(mpm_merge_local(A, NULL, NULL, NULL, 2, 64, 64, MPM_BF16, 8, -1, 0, A2, A2, NULL, A2, A2, A, big, NULL, NULL,
                           NULL), MPM_ERR_INVALID_ARG);                                 /* window < 0 */
    EXPECT(mpm_merge_local(A, NULL, NULL, NULL, 2, 64, 64, MPM_BF16, 8, 1, 64, A2, A2, NULL, A2, A2, A, big, NULL, NULL,
                           NULL), MPM_ERR_INVALID_ARG);                                 /* block_rows */
    EXPECT(mpm_merge_local(A, NULL, A, NULL, 2, 64, 40, MPM_BF16, 8, 1, 0, A2, A2, NULL, A2, A2, A, big, NULL, NULL,
                           NULL), MPM_ERR_UNSUPPORTED);                                 /* norms, 80-byte rows */
    EXPECT(mpm_merge_local(A, NULL, NULL, NULL, 2, 64, 64, MPM_BF16, 8, 1, 0, A2, A2, NULL, A2, A2, A, 16, NULL, NULL,
                           NULL), MPM_ERR_WORKSPACE);
    {
        int32_t rows = -7;
        EXPECT(mpm_local_block_rows(2, 64, 64, MPM_BF16, 8, 1, 0, NULL), MPM_ERR_INVALID_ARG);
        EXPECT(mpm_local_block_rows(2, 64, 64, MPM_BF16, 8, 1, 100, &rows), MPM_ERR_INVALID_ARG);
        EXPECT(mpm_local_block_rows(2, 64, 64, MPM_BF16, MPM_MAX_N + 1, 1, 0, &rows), MPM_ERR_INVALID_ARG);
        if (rows != -7) return 1;
    }
    EXPECT(mpm_pad(A, A2, 2, 8, 40, A, NULL), MPM_ERR_INVALID_ARG);
    EXPECT(mpm_unpad(A, NULL, 2, 8, 64, A, NULL), MPM_ERR_INVALID_ARG);
    EXPECT(mpm_last_hip_error(), 0);
    if (mpm_status_string(42) == NULL || strcmp(mpm_status_string(MPM_ERR_HIP), "MPM_ERR_HIP") != 0) return 1;

    if (inject) {
        /* Valid arguments: every launching entry point reports the injected failure. */
        const int hip_launch_failure = 719;  /* hipErrorLaunchFailure */
        EXPECT(mpm_workspace_init(A, big, NULL), MPM_ERR_HIP);
        EXPECT(mpm_last_hip_error(), hip_launch_failure);
        EXPECT(mpm_affinity(A, NULL, NULL, 2, 16, 64, MPM_BF16, 0, A, big, NULL, NULL, NULL), MPM_ERR_HIP);
        EXPECT(mpm_affinity_compact(A, NULL, NULL, 2, 16, 64, MPM_BF16, 0, A2, A2, A, big, NULL, NULL, NULL),
               MPM_ERR_HIP);
        EXPECT(mpm_argmax(A, NULL, 2, 16, 64, MPM_BF16, 0, A2, NULL, A, big, NULL), MPM_ERR_HIP);
        EXPECT(mpm_pair_compact(A, NULL, 2, 16, A2, A2, A2, NULL), MPM_ERR_HIP);
        EXPECT(mpm_pair_average(A, NULL, A2, A2, 2, 16, 64, MPM_BF16, A2, NULL, NULL), MPM_ERR_HIP);
        EXPECT(mpm_merge(A, NULL, NULL, 2, 16, 64, MPM_BF16, 0, A2, A2, NULL, A2, A, big, NULL), MPM_ERR_HIP);
        EXPECT(mpm_merge_noalloc(A, NULL, NULL, 2, 16, 64, MPM_BF16, 0, A2, A2, NULL, A2, NULL), MPM_ERR_HIP);
        EXPECT(mpm_compose(A, A2, 2, 16, A, NULL), MPM_ERR_HIP);
        EXPECT(mpm_unmerge(A, NULL, A2, NULL, 0, 2, 16, 64, MPM_BF16, A, NULL), MPM_ERR_HIP);
        EXPECT(mpm_compose_unmerge(A, NULL, A2, A2, NULL, NULL, 0, 2, 16, 64, MPM_BF16, A, NULL), MPM_ERR_HIP);
        EXPECT(mpm_merge_local(A, NULL, NULL, NULL, 2, 64, 64, MPM_BF16, 8, 1, 0, A2, A2, NULL, A2, A2, A, big, NULL,
                               NULL, NULL), MPM_ERR_HIP);
        EXPECT(mpm_pad(A, A2, 2, 8, 64, A, NULL), MPM_ERR_HIP);
        EXPECT(mpm_unpad(A, A2, 2, 8, 64, A, NULL), MPM_ERR_HIP);
        EXPECT(mpm_last_hip_error(), hip_launch_failure);
    }
    printf("abi driver: ok%s\n", inject ? " (with injected launch failures)" : "");
    return 0;
}
