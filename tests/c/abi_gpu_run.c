/* A plain C client of the full hot path on the GPU: reads a segment table
 * and its rows from a directory, allocates device memory with the HIP C
 * API, calls msao_run (statistics, MAS, selection, compaction) on the null
 * stream and writes every output array to another directory. No Python and
 * no framework: only include/msao.h, libmsao.so and the HIP runtime.
 * Built by the package's build step; tests/test_gpu_c_client.py runs it and
 * compares its outputs with the oracle.
 *
 * usage: abi_gpu_run IN_DIR OUT_DIR
 *   IN_DIR/segments.txt: "n R flags", then per segment
 *   "request modality n_frames tokens_per_frame hidden dtype keep_ratio file"
 *   with the file holding the segment's rows (row stride = hidden).
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "msao.h"

#define MAX_SEGS 64

#define HIP_OK(call)                                                                    \
    do {                                                                                \
        hipError_t e_ = (call);                                                         \
        if (e_ != hipSuccess) {                                                         \
            fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));           \
            exit(3);                                                                    \
        }                                                                               \
    } while (0)

static void* dalloc(size_t bytes)
{
    void* p = NULL;
    HIP_OK(hipMalloc(&p, bytes ? bytes : 256));
    HIP_OK(hipMemset(p, 0, bytes ? bytes : 256));
    return p;
}

static void dump(const char* dir, const char* name, const void* dev, size_t bytes)
{
    char path[1024];
    snprintf(path, sizeof path, "%s/%s", dir, name);
    void* h = malloc(bytes ? bytes : 1);
    if (!h) exit(2);
    if (bytes) HIP_OK(hipMemcpy(h, dev, bytes, hipMemcpyDeviceToHost));
    FILE* f = fopen(path, "wb");
    if (!f) exit(2);
    if (bytes && fwrite(h, 1, bytes, f) != bytes) exit(2);
    fclose(f);
    free(h);
}

int main(int argc, char** argv)
{
    if (argc != 3) {
        fprintf(stderr, "usage: %s IN_DIR OUT_DIR\n", argv[0]);
        return 2;
    }
    char path[1024];
    snprintf(path, sizeof path, "%s/segments.txt", argv[1]);
    FILE* f = fopen(path, "r");
    if (!f) return 2;
    int n = 0, R = 0;
    unsigned flags = 0;
    if (fscanf(f, "%d %d %u", &n, &R, &flags) != 3 || n < 0 || n > MAX_SEGS) return 2;
    msao_segment segs[MAX_SEGS];
    for (int i = 0; i < n; ++i) {
        char file[512];
        msao_segment* s = &segs[i];
        memset(s, 0, sizeof *s);
        if (fscanf(f, "%d %d %d %d %d %d %f %511s", &s->request, &s->modality, &s->n_frames,
                   &s->tokens_per_frame, &s->hidden, &s->dtype, &s->keep_ratio, file) != 8)
            return 2;
        s->row_stride = s->hidden;
        const size_t es = s->dtype == MSAO_F32 ? 4 : 2;
        const size_t bytes = (size_t)s->n_frames * (size_t)s->tokens_per_frame * (size_t)s->hidden * es;
        snprintf(path, sizeof path, "%s/%s", argv[1], file);
        FILE* g = fopen(path, "rb");
        if (!g) return 2;
        void* h = malloc(bytes ? bytes : 1);
        if (!h || (bytes && fread(h, 1, bytes, g) != bytes)) return 2;
        fclose(g);
        void* d = dalloc(bytes);
        if (bytes) HIP_OK(hipMemcpy(d, h, bytes, hipMemcpyHostToDevice));
        free(h);
        s->data = d;
    }
    fclose(f);

    msao_params p = msao_default_params();
    p.flags = flags;
    msao_status st = msao_validate(segs, n, R, &p);
    if (st != MSAO_OK) {
        fprintf(stderr, "validate: %s: %s\n", msao_status_string(st), msao_last_error_global());
        return 4;
    }
    int64_t nt = 0, nf = 0;
    size_t ws_bytes = 0;
    int64_t off[MAX_SEGS], out_bytes = 0;
    if (msao_count(segs, n, &nt, &nf) != MSAO_OK || msao_workspace_size(segs, n, R, &ws_bytes) != MSAO_OK ||
        msao_compact_layout(segs, n, off, &out_bytes) != MSAO_OK)
        return 4;
    const size_t T = (size_t)nt, F = (size_t)nf, X = (size_t)R * MSAO_NUM_MODALITIES;
    msao_token_out tok = {dalloc(4 * T), dalloc(4 * T), dalloc(4 * T), dalloc(4 * T), dalloc(4 * T), dalloc(4 * T)};
    msao_frame_out frm = {dalloc(8 * F), dalloc(4 * F), dalloc(4 * F)};
    msao_req_out req = {dalloc(8 * 4 * X), dalloc(4 * X), dalloc(4 * X), dalloc(4 * X), dalloc(4 * X), dalloc(X)};
    msao_select_out sel = {dalloc(T), dalloc(4 * T), dalloc(4 * (size_t)(n > 0 ? n : 1))};
    void* out = dalloc((size_t)out_bytes);
    void* ws = dalloc(ws_bytes);

    msao_ctx* ctx = NULL;
    st = msao_create(&ctx, 0);
    if (st != MSAO_OK) {
        fprintf(stderr, "create: %s\n", msao_last_error_global());
        return 4;
    }
    st = msao_run(ctx, segs, n, R, &p, NULL, &tok, &frm, &req, &sel, out, off, out_bytes, ws, ws_bytes, NULL);
    if (st != MSAO_OK) {
        fprintf(stderr, "run: %s: %s\n", msao_status_string(st), msao_last_error(ctx));
        return 4;
    }
    HIP_OK(hipDeviceSynchronize());

    const char* o = argv[2];
    dump(o, "z.bin", tok.z, 4 * T);
    dump(o, "l1.bin", tok.l1, 4 * T);
    dump(o, "l2.bin", tok.l2, 4 * T);
    dump(o, "d.bin", tok.d, 4 * T);
    dump(o, "dframe.bin", frm.dframe, 8 * F);
    dump(o, "sim.bin", frm.sim, 4 * F);
    dump(o, "agg.bin", req.agg, 8 * 4 * X);
    dump(o, "mas.bin", req.mas, 4 * X);
    dump(o, "keep.bin", sel.keep, T);
    dump(o, "kept_idx.bin", sel.kept_idx, 4 * T);
    dump(o, "kept_count.bin", sel.kept_count, 4 * (size_t)n);
    dump(o, "out.bin", out, (size_t)out_bytes);
    snprintf(path, sizeof path, "%s/offsets.bin", o);
    FILE* fo = fopen(path, "wb");
    if (!fo || fwrite(off, sizeof(int64_t), (size_t)n, fo) != (size_t)n) return 2;
    fclose(fo);
    msao_destroy(ctx);
    printf("ok: %d segments, %lld tokens, %lld frames\n", n, (long long)nt, (long long)nf);
    return 0;
}
