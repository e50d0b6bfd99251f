/* Calls the scan through the C-ABI from plain C (HIP runtime API for device
 * memory, no other framework): reads A, b, lambda_K (float32) from a file,
 * runs lbi_scan_backward (the library's choice, workspace included) and
 * lbi_scan_backward_ex with LBI_ALGO_CHAIN, and writes both lambda arrays.
 * Usage: scan_from_c IN OUT B K r */
#include <stdio.h>
#include <stdlib.h>

#include <hip/hip_runtime_api.h>

#include "lbi.h"

#define HIP_OK(call)                                                                  \
    do {                                                                              \
        hipError_t e_ = (call);                                                       \
        if (e_ != hipSuccess) {                                                       \
            fprintf(stderr, "%s: %s\n", #call, hipGetErrorString(e_));                \
            return 2;                                                                 \
        }                                                                             \
    } while (0)

int main(int argc, char **argv)
{
    if (argc != 6) {
        fprintf(stderr, "usage: %s IN OUT B K r\n", argv[0]);
        return 1;
    }
    const long B = atol(argv[3]), K = atol(argv[4]);
    const int r = atoi(argv[5]);
    const size_t nA = (size_t)B * K * r * r, nb = (size_t)B * K * r, nl = (size_t)B * r;
    float *host = malloc((nA + nb + nl) * sizeof(float));
    float *out = malloc(2 * nb * sizeof(float));
    FILE *f = fopen(argv[1], "rb");
    if (!host || !out || !f || fread(host, sizeof(float), nA + nb + nl, f) != nA + nb + nl) {
        fprintf(stderr, "cannot read %s\n", argv[1]);
        return 1;
    }
    fclose(f);

    void *dA, *db, *dl, *dlam, *dlam2, *ws = NULL;
    HIP_OK(hipMalloc(&dA, nA * sizeof(float)));
    HIP_OK(hipMalloc(&db, nb * sizeof(float)));
    HIP_OK(hipMalloc(&dl, nl * sizeof(float)));
    HIP_OK(hipMalloc(&dlam, nb * sizeof(float)));
    HIP_OK(hipMalloc(&dlam2, nb * sizeof(float)));
    HIP_OK(hipMemcpy(dA, host, nA * sizeof(float), hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(db, host + nA, nb * sizeof(float), hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dl, host + nA + nb, nl * sizeof(float), hipMemcpyHostToDevice));

    const size_t wsb = lbi_scan_backward_workspace_bytes(B, K, r, LBI_F32);
    if (wsb > 0)
        HIP_OK(hipMalloc(&ws, wsb));
    lbi_status st = lbi_scan_backward(dA, db, dl, (float *)dlam, B, K, r, LBI_F32, ws, wsb, NULL);
    if (st != LBI_OK) {
        fprintf(stderr, "lbi_scan_backward: %s\n", lbi_status_string(st));
        return 3;
    }
    st = lbi_scan_backward_ex(dA, db, dl, (float *)dlam2, B, K, r, LBI_F32, NULL, 0, NULL, NULL,
                              LBI_MATH_DEFAULT, LBI_ALGO_CHAIN);
    if (st != LBI_OK) {
        fprintf(stderr, "lbi_scan_backward_ex: %s\n", lbi_status_string(st));
        return 3;
    }
    HIP_OK(hipDeviceSynchronize());
    HIP_OK(hipMemcpy(out, dlam, nb * sizeof(float), hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(out + nb, dlam2, nb * sizeof(float), hipMemcpyDeviceToHost));
    f = fopen(argv[2], "wb");
    if (!f || fwrite(out, sizeof(float), 2 * nb, f) != 2 * nb) {
        fprintf(stderr, "cannot write %s\n", argv[2]);
        return 1;
    }
    fclose(f);
    printf("workspace %zu bytes\n", wsb);
    hipFree(dA);
    hipFree(db);
    hipFree(dl);
    hipFree(dlam);
    hipFree(dlam2);
    if (ws)
        hipFree(ws);
    free(host);
    free(out);
    return 0;
}
