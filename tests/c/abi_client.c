/* A plain C client of libiefwd (no Python, no torch): creates an instance of
 * a two-layer post-LN encoder, puts it on a 64-CU quota, submits one batch
 * from host memory, reads the logits back and writes them, fp32 in C order,
 * to the file named by argv[1].  The input is x[i] = ((i * 7919) mod 2001 -
 * 1000) / 1000 over the batch's B * S * d elements, an exact fp32 expression
 * that any client can reproduce.
 *
 * Exit status: 0 on success, 2 on bad usage, 3 with the library's status
 * string and message on stderr if a call fails (ENODEV without a GPU). */
#include <stdio.h>
#include <stdlib.h>

#include "iefwd.h"

#define B 2u
#define S 32u
#define D 128u
#define N_OUT 2u

static int fail(const char *what, int st) {
    fprintf(stderr, "%s: %s (%d): %s\n", what, iefwd_status_string(st), st, iefwd_last_error());
    return 3;
}

int main(int argc, char **argv) {
    if (argc != 2) {
        fprintf(stderr, "usage: %s OUT_FILE\n", argv[0]);
        return 2;
    }
    iefwd_config cfg;
    iefwd_config_init(&cfg);
    cfg.n_layers = 2;
    cfg.d_model = D;
    cfg.n_heads = 2;
    cfg.d_ff = 512;
    cfg.max_batch = B;
    cfg.max_seq = S;
    cfg.n_out = N_OUT;
    cfg.seed = 7;

    iefwd_instance *inst = NULL;
    int st = iefwd_create(&cfg, 0, &inst);
    if (st != IEFWD_OK) return fail("iefwd_create", st);

    static float x[B * S * D], logits[B * S * N_OUT];
    for (unsigned i = 0; i < B * S * D; ++i) x[i] = (float)((int)((i * 7919u) % 2001u) - 1000) / 1000.0f;

    int rc = 0;
    if ((st = iefwd_set_quota(inst, 64)) != IEFWD_OK) rc = fail("iefwd_set_quota", st);
    else if ((st = iefwd_submit(inst, x, B, S, 0)) != IEFWD_OK) rc = fail("iefwd_submit", st);
    else if ((st = iefwd_read_logits(inst, logits, B * S * N_OUT, 0)) != IEFWD_OK) rc = fail("iefwd_read_logits", st);
    if (rc == 0) {
        FILE *f = fopen(argv[1], "wb");
        if (!f || fwrite(logits, sizeof logits, 1, f) != 1) {
            fprintf(stderr, "cannot write %s\n", argv[1]);
            rc = 3;
        }
        if (f) fclose(f);
    }
    iefwd_destroy(inst);
    return rc;
}
