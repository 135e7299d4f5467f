/*
 * Plain C user of the f3s C ABI (include/f3s.h): no Python, no torch.
 *
 * usage: f3s_c_driver DIR N NNZ D SCALE
 *   DIR/row_ptr.bin  int32[N+1]      DIR/col_idx.bin  int32[NNZ]
 *   DIR/q.bin, k.bin, v.bin          binary16 [N, D] row-major
 * writes DIR/o.bin (fp32 [N, D]) and DIR/info.txt (plan statistics and the
 * results of the argument-error checks), exits 0 on success.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "f3s.h"

#define HIP_OK(x)                                                              \
    do {                                                                       \
        hipError_t e_ = (x);                                                   \
        if (e_ != hipSuccess) {                                                \
            fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));    \
            return 2;                                                          \
        }                                                                      \
    } while (0)

static void *read_file(const char *dir, const char *name, size_t bytes)
{
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", dir, name);
    FILE *f = fopen(path, "rb");
    if (!f) return NULL;
    void *buf = malloc(bytes ? bytes : 1);
    if (buf && fread(buf, 1, bytes, f) != bytes) {
        free(buf);
        buf = NULL;
    }
    fclose(f);
    return buf;
}

static void *to_device(const void *host, size_t bytes)
{
    void *d = NULL;
    if (hipMalloc(&d, bytes ? bytes : 16) != hipSuccess) return NULL;
    if (bytes && hipMemcpy(d, host, bytes, hipMemcpyHostToDevice) != hipSuccess) {
        (void)hipFree(d);
        return NULL;
    }
    return d;
}

int main(int argc, char **argv)
{
    if (argc != 6) {
        fprintf(stderr, "usage: %s DIR N NNZ D SCALE\n", argv[0]);
        return 1;
    }
    const char *dir = argv[1];
    const int32_t N = (int32_t)atol(argv[2]);
    const size_t nnz = (size_t)atoll(argv[3]);
    const int32_t d = (int32_t)atol(argv[4]);
    const float scale = (float)atof(argv[5]);
    const size_t feat = (size_t)N * (size_t)d;

    int32_t *rp = read_file(dir, "row_ptr.bin", sizeof(int32_t) * ((size_t)N + 1));
    int32_t *ci = read_file(dir, "col_idx.bin", sizeof(int32_t) * nnz);
    void *q = read_file(dir, "q.bin", 2 * feat);
    void *k = read_file(dir, "k.bin", 2 * feat);
    void *v = read_file(dir, "v.bin", 2 * feat);
    if (!rp || !ci || !q || !k || !v) {
        fprintf(stderr, "cannot read the inputs in %s\n", dir);
        return 1;
    }
    int32_t *d_rp = to_device(rp, sizeof(int32_t) * ((size_t)N + 1));
    int32_t *d_ci = to_device(ci, sizeof(int32_t) * nnz);
    void *d_q = to_device(q, 2 * feat), *d_k = to_device(k, 2 * feat), *d_v = to_device(v, 2 * feat);
    float *d_o = NULL;
    HIP_OK(hipMalloc((void **)&d_o, 4 * (feat ? feat : 4)));
    if (!d_rp || !d_ci || !d_q || !d_k || !d_v) {
        fprintf(stderr, "device allocation failed\n");
        return 2;
    }

    char path[4096];
    snprintf(path, sizeof path, "%s/info.txt", dir);
    FILE *info = fopen(path, "w");
    if (!info) return 1;

    /* the plan (Section 3.1 layout, Section 3.2 work list) */
    f3s_plan_t plan = f3s_plan(d_rp, d_ci, N);
    if (!plan) {
        fprintf(stderr, "f3s_plan: %s\n", f3s_status_string(f3s_last_error()));
        return 3;
    }
    f3s_plan_info_t pi;
    if (f3s_plan_info(plan, &pi) != F3S_OK) return 3;
    fprintf(info, "n_windows %d\nnnz %lld\nn_blocks %lld\nn_items %d\nn_split %d\n",
            pi.n_windows, (long long)pi.nnz, (long long)pi.n_blocks, pi.n_items, pi.n_split);

    /* the fused operator on the null stream */
    f3s_status_t st = f3s_run(plan, d_q, d_k, d_v, d_o, d, scale, NULL);
    if (st != F3S_OK) {
        fprintf(stderr, "f3s_run: %s\n", f3s_status_string(st));
        return 4;
    }
    HIP_OK(hipDeviceSynchronize());
    float *o = malloc(4 * (feat ? feat : 1));
    HIP_OK(hipMemcpy(o, d_o, 4 * feat, hipMemcpyDeviceToHost));
    snprintf(path, sizeof path, "%s/o.bin", dir);
    FILE *fo = fopen(path, "wb");
    if (!fo || fwrite(o, 4, feat, fo) != feat) return 1;
    fclose(fo);

    /* the same plan built into a caller-lent workspace gives the same O */
    const size_t ws_bytes = f3s_plan_workspace_bytes(N, (int64_t)nnz);
    void *d_ws = NULL;
    HIP_OK(hipMalloc(&d_ws, ws_bytes ? ws_bytes : 256));
    f3s_plan_t plan_ws = f3s_plan_ws(d_rp, d_ci, N, d_ws, ws_bytes);
    if (!plan_ws) {
        fprintf(stderr, "f3s_plan_ws: %s\n", f3s_status_string(f3s_last_error()));
        return 3;
    }
    float *d_o2 = NULL;
    HIP_OK(hipMalloc((void **)&d_o2, 4 * (feat ? feat : 4)));
    st = f3s_run(plan_ws, d_q, d_k, d_v, d_o2, d, scale, NULL);
    HIP_OK(hipDeviceSynchronize());
    float *o2 = malloc(4 * (feat ? feat : 1));
    HIP_OK(hipMemcpy(o2, d_o2, 4 * feat, hipMemcpyDeviceToHost));
    fprintf(info, "ws_run %s same %d\n", f3s_status_string(st),
            feat == 0 || memcmp(o, o2, 4 * feat) == 0);
    f3s_plan_t short_ws = f3s_plan_ws(d_rp, d_ci, N, d_ws, ws_bytes / 2);
    fprintf(info, "ws_short %s %s\n", short_ws ? "plan" : "null",
            f3s_status_string(f3s_last_error()));
    f3s_destroy(short_ws);
    f3s_destroy(plan_ws);
    (void)hipFree(d_ws);
    (void)hipFree(d_o2);
    free(o2);

    /* windows aligned to graphs of 7 rows each (f3s_plan_segments, host
       offsets): same operator, so O again within the parity bar */
    {
        const int32_t n_segs = (N + 6) / 7;
        int32_t *seg = malloc(sizeof(int32_t) * ((size_t)n_segs + 1));
        for (int32_t g = 0; g <= n_segs; ++g) seg[g] = g * 7 < N ? g * 7 : N;
        f3s_plan_t sp = f3s_plan_segments(d_rp, d_ci, N, seg, n_segs);
        if (!sp) {
            fprintf(stderr, "f3s_plan_segments: %s\n", f3s_status_string(f3s_last_error()));
            return 3;
        }
        f3s_plan_info_t si;
        if (f3s_plan_info(sp, &si) != F3S_OK) return 3;
        int32_t *wr = malloc(sizeof(int32_t) * ((size_t)si.n_windows + 1));
        if (f3s_plan_window_rows(sp, wr) != F3S_OK) return 3;
        fprintf(info, "seg_windows %d first %d %d %d last %d\n", si.n_windows,
                wr[0], si.n_windows > 0 ? wr[1] : -1, si.n_windows > 1 ? wr[2] : -1,
                wr[si.n_windows]);
        st = f3s_run(sp, d_q, d_k, d_v, d_o, d, scale, NULL);
        HIP_OK(hipDeviceSynchronize());
        float *os = malloc(4 * (feat ? feat : 1));
        HIP_OK(hipMemcpy(os, d_o, 4 * feat, hipMemcpyDeviceToHost));
        snprintf(path, sizeof path, "%s/o_seg.bin", dir);
        FILE *fs = fopen(path, "wb");
        if (!fs || fwrite(os, 4, feat, fs) != feat) return 1;
        fclose(fs);
        fprintf(info, "seg_run %s\n", f3s_status_string(st));
        f3s_destroy(sp);
        free(wr);
        free(os);
        free(seg);
    }

    /* argument errors are reported, not launched */
    st = f3s_run(plan, d_q, d_k, d_v, d_o, d + 8, scale, NULL);
    fprintf(info, "bad_d %s\n", f3s_status_string(st));
    st = f3s_run(NULL, d_q, d_k, d_v, d_o, d, scale, NULL);
    fprintf(info, "null_plan %s last_error %s\n", f3s_status_string(st),
            f3s_status_string(f3s_last_error()));
    st = f3s_run(plan, d_q, d_k, d_v, (char *)d_o + 4, d, scale, NULL);
    fprintf(info, "misaligned_out %s\n", f3s_status_string(st));
    int32_t bad_rp[3] = {0, 2, 1};   /* decreasing row pointer */
    int32_t *d_bad = to_device(bad_rp, sizeof bad_rp);
    f3s_plan_t bad = f3s_plan(d_bad, d_ci, 2);
    fprintf(info, "bad_csr %s %s\n", bad ? "plan" : "null",
            f3s_status_string(f3s_last_error()));
    f3s_destroy(bad);
    f3s_destroy(plan);
    f3s_destroy(NULL);
    fclose(info);
    (void)hipFree(d_bad);
    (void)hipFree(d_rp);
    (void)hipFree(d_ci);
    (void)hipFree(d_q);
    (void)hipFree(d_k);
    (void)hipFree(d_v);
    (void)hipFree(d_o);
    free(rp);
    free(ci);
    free(q);
    free(k);
    free(v);
    free(o);
    return 0;
}
