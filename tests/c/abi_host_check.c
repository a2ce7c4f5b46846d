/* A plain C client of the library's host-only entry points (no GPU needed):
 * segment-table validation and sizes, then Algorithm 1's threshold logic
 * (Sec. 4.2) over normalised entropies read from a file. Used by
 * tests/test_abi_c_client.py, which builds it with gcc against
 * include/msao.h and checks what it prints and writes against the oracle.
 *
 * usage: abi_host_check ENTROPIES.f32 N_CALIB DECISIONS.i8 THETAS.f64
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "msao.h"

static int check(msao_status got, msao_status want, const char* what)
{
    if (got != want) {
        printf("FAIL %s: %s (want %s)\n", what, msao_status_string(got), msao_status_string(want));
        return 1;
    }
    return 0;
}

int main(int argc, char** argv)
{
    if (argc != 5) {
        fprintf(stderr, "usage: %s ENTROPIES.f32 N_CALIB DECISIONS.i8 THETAS.f64\n", argv[0]);
        return 2;
    }
    int bad = 0;
    /* a tri-modal request: the data pointers are only checked, never read */
    static _Alignas(16) uint16_t storage[8];
    msao_segment segs[3] = {
        {storage, 1024, 0, MSAO_IMAGE, 1, 576, 1024, MSAO_BF16, 0.25f},
        {storage, 1280, 0, MSAO_AUDIO, 1, 1500, 1280, MSAO_BF16, 0.5f},
        {storage, 4096, 0, MSAO_TEXT, 1, 128, 4096, MSAO_BF16, 1.0f},
    };
    msao_params p = msao_default_params();
    bad |= check(msao_validate(segs, 3, 1, &p), MSAO_OK, "validate");
    int64_t nt = 0, nf = 0;
    bad |= check(msao_count(segs, 3, &nt, &nf), MSAO_OK, "count");
    size_t ws = 0;
    bad |= check(msao_workspace_size(segs, 3, 1, &ws), MSAO_OK, "workspace_size");
    int64_t off[3], total = 0;
    bad |= check(msao_compact_layout(segs, 3, off, &total), MSAO_OK, "compact_layout");
    printf("tokens %lld frames %lld workspace %zu layout %lld %lld %lld total %lld\n", (long long)nt, (long long)nf,
           ws, (long long)off[0], (long long)off[1], (long long)off[2], (long long)total);
    /* errors: a ragged bf16 width, an unknown flag bit, a request id out of range */
    segs[0].hidden = 1020;
    bad |= check(msao_validate(segs, 3, 1, &p), MSAO_ERR_ALIGNMENT, "ragged width");
    segs[0].hidden = 1024;
    p.flags = 0x80u;
    bad |= check(msao_validate(segs, 3, 1, &p), MSAO_ERR_INVALID_ARG, "flag bits");
    p.flags = MSAO_FLAG_SELECT_PER_FRAME;
    bad |= check(msao_validate(segs, 3, 1, &p), MSAO_OK, "per-frame flag");
    segs[2].request = 1;
    bad |= check(msao_validate(segs, 3, 1, &p), MSAO_ERR_INVALID_ARG, "request id");
    printf("last error: %s\n", msao_last_error_global());

    /* Algorithm 1 over the entropies */
    FILE* f = fopen(argv[1], "rb");
    if (!f) return 2;
    fseek(f, 0, SEEK_END);
    const long n = ftell(f) / (long)sizeof(float);
    fseek(f, 0, SEEK_SET);
    float* h = (float*)malloc(sizeof(float) * (size_t)n);
    if (!h || fread(h, sizeof(float), (size_t)n, f) != (size_t)n) return 2;
    fclose(f);
    const int64_t ncal = atoll(argv[2]);
    msao_sched_params sp = msao_sched_default_params();
    msao_sched_state st;
    bad |= check(msao_sched_init(h, ncal, &sp, &st), MSAO_OK, "sched_init");
    printf("theta0 %.17g p_conf %.17g n_draft %d\n", st.theta, st.p_conf, st.n_draft);
    int8_t* dec = (int8_t*)malloc((size_t)n);
    double* th = (double*)malloc(sizeof(double) * (size_t)n);
    bad |= check(msao_sched_run(&st, &sp, h, n, dec, th), MSAO_OK, "sched_run");
    printf("steps %lld held %lld sends %lld offloads %lld tokens_sent %lld\n", (long long)st.steps,
           (long long)st.held, (long long)st.sends, (long long)st.offloads, (long long)st.tokens_sent);
    FILE* fd = fopen(argv[3], "wb");
    FILE* ft = fopen(argv[4], "wb");
    if (!fd || !ft) return 2;
    fwrite(dec, 1, (size_t)n, fd);
    fwrite(th, sizeof(double), (size_t)n, ft);
    fclose(fd);
    fclose(ft);
    /* the latency model (Eq. 8, 13, 14) and the retention floor */
    const double spec = msao_expected_spec_tokens(st.p_conf);
    const double comm = msao_comm_latency(2.0e6, 1.25e7, 0.02);
    float mas[2] = {0.25f, 0.75f}, beta[2] = {0, 0};
    bad |= check(msao_retention_floor(mas, 2, beta), MSAO_OK, "retention_floor");
    printf("spec %.17g comm %.17g beta %.9g %.9g\n", spec, comm, beta[0], beta[1]);
    free(h);
    free(dec);
    free(th);
    printf(bad ? "FAILED\n" : "OK\n");
    return bad;
}
