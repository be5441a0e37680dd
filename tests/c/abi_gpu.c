/* A C client of libreshard.so on the GPU, with no Python and no torch in the
 * process: device memory, copies and the stream come from the HIP runtime
 * directly.
 *
 *     abi_gpu CASE SRC_BIN DST_BIN
 *
 * CASE is a text file of lines "key value...":
 *     dtype  <reshard_dtype_t code>
 *     shape  <ndim> <d0> ...
 *     src    <mesh ndim> <m0> ... <spec>      (spec without blanks, e.g. R,S^1,R)
 *     dst    <mesh ndim> <m0> ... <spec>
 *     block  <threads per workgroup, 0 = default>
 *     stream <0: the null stream, 1: a created stream>
 *     upload <0 or 1: call reshard_plan_upload before executing>
 *     repeat <executes of the plan, >= 1>
 *     flags  <reshard_plan flags, default 0>
 * SRC_BIN holds the source shards back to back in device order (each the
 * dense C-order local shard).  The program plans, copies the shards to
 * device buffers, fills the destination buffers with 0xA5, executes, and
 * writes the destination shards back to back to DST_BIN.  Each buffer is
 * allocated with 256 guard bytes on both sides, filled with 0x5A, which
 * must be untouched afterwards; the sources must be unmodified.  Prints
 * "ok" and exits 0 on success. */
#include <inttypes.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "reshard.h"

#define GUARD 256

#define FAIL(...)                             \
    do {                                      \
        fprintf(stderr, __VA_ARGS__);         \
        fputc('\n', stderr);                  \
        return 1;                             \
    } while (0)
#define HIPCHECK(x)                                                                   \
    do {                                                                              \
        hipError_t e_ = (x);                                                          \
        if (e_ != hipSuccess) FAIL("%s: %s", #x, hipGetErrorString(e_));              \
    } while (0)
#define RSCHECK(x)                                                                    \
    do {                                                                              \
        reshard_status_t s_ = (x);                                                    \
        if (s_ != RESHARD_OK) FAIL("%s: status %d: %s", #x, (int)s_, reshard_last_error()); \
    } while (0)

typedef struct {
    int mesh_ndim;
    int64_t mesh[RESHARD_MAX_MESH_NDIM];
    char spec[256];
} side_t;

static int read_side(FILE *f, side_t *s) {
    if (fscanf(f, "%d", &s->mesh_ndim) != 1 || s->mesh_ndim < 1 || s->mesh_ndim > RESHARD_MAX_MESH_NDIM) return 0;
    for (int i = 0; i < s->mesh_ndim; ++i)
        if (fscanf(f, "%" SCNd64, &s->mesh[i]) != 1) return 0;
    return fscanf(f, "%255s", s->spec) == 1;
}

static int64_t product(const int64_t *v, int n) {
    int64_t p = 1;
    for (int i = 0; i < n; ++i) p *= v[i];
    return p;
}

static const size_t kElemSize[] = {1, 1, 2, 2, 4, 4, 8, 8, 2, 2, 4, 8};

int main(int argc, char **argv) {
    if (argc != 4) FAIL("usage: abi_gpu CASE SRC_BIN DST_BIN");
    FILE *f = fopen(argv[1], "r");
    if (!f) FAIL("cannot open %s", argv[1]);
    int dtype = -1, ndim = 0, block = 0, use_stream = 0, upload = 0, repeat = 1;
    unsigned flags = 0;
    int64_t shape[RESHARD_MAX_NDIM];
    side_t src, dst;
    char key[32];
    while (fscanf(f, "%31s", key) == 1) {
        int ok = 1;
        if (!strcmp(key, "dtype")) ok = fscanf(f, "%d", &dtype) == 1;
        else if (!strcmp(key, "shape")) {
            ok = fscanf(f, "%d", &ndim) == 1 && ndim >= 1 && ndim <= RESHARD_MAX_NDIM;
            for (int i = 0; ok && i < ndim; ++i) ok = fscanf(f, "%" SCNd64, &shape[i]) == 1;
        } else if (!strcmp(key, "src")) ok = read_side(f, &src);
        else if (!strcmp(key, "dst")) ok = read_side(f, &dst);
        else if (!strcmp(key, "block")) ok = fscanf(f, "%d", &block) == 1;
        else if (!strcmp(key, "stream")) ok = fscanf(f, "%d", &use_stream) == 1;
        else if (!strcmp(key, "upload")) ok = fscanf(f, "%d", &upload) == 1;
        else if (!strcmp(key, "repeat")) ok = fscanf(f, "%d", &repeat) == 1 && repeat >= 1;
        else if (!strcmp(key, "flags")) ok = fscanf(f, "%u", &flags) == 1;
        else ok = 0;
        if (!ok) FAIL("bad case line at key %s", key);
    }
    fclose(f);
    if (dtype < 0 || dtype > 11 || ndim == 0) FAIL("case needs dtype and shape");
    const size_t es = kElemSize[dtype];

    reshard_tuning_t tun;
    memset(&tun, 0, sizeof tun);
    tun.block_threads = block;
    reshard_plan_t *plan = NULL;
    RSCHECK(reshard_plan_ex(ndim, shape, (reshard_dtype_t)dtype, src.mesh_ndim, src.mesh, src.spec, dst.mesh_ndim,
                            dst.mesh, dst.spec, flags, &tun, &plan));

    const int64_t nsrc = product(src.mesh, src.mesh_ndim), ndst = product(dst.mesh, dst.mesh_ndim);
    size_t *sbytes = calloc((size_t)nsrc, sizeof *sbytes), *dbytes = calloc((size_t)ndst, sizeof *dbytes);
    unsigned char **sraw = calloc((size_t)nsrc, sizeof *sraw), **draw = calloc((size_t)ndst, sizeof *draw);
    void **sp = calloc((size_t)nsrc, sizeof *sp), **dp = calloc((size_t)ndst, sizeof *dp);
    if (!sbytes || !dbytes || !sraw || !draw || !sp || !dp) FAIL("out of host memory");
    size_t stotal = 0, dtotal = 0, maxb = 0;
    for (int64_t k = 0; k < nsrc + ndst; ++k) {
        const int side = k < nsrc ? 0 : 1;
        const int64_t dev = side ? k - nsrc : k;
        int64_t ls[RESHARD_MAX_NDIM];
        RSCHECK(reshard_plan_local_shape(plan, side, dev, ls));
        const size_t b = (size_t)product(ls, ndim) * es;
        if (side) dbytes[dev] = b, dtotal += b;
        else sbytes[dev] = b, stotal += b;
        if (b > maxb) maxb = b;
    }

    unsigned char *host = malloc(maxb + 2 * GUARD + 1);
    unsigned char *sall = malloc(stotal + 1), *dall = malloc(dtotal + 1);
    if (!host || !sall || !dall) FAIL("out of host memory");
    f = fopen(argv[2], "rb");
    if (!f || fread(sall, 1, stotal, f) != stotal) FAIL("cannot read %zu source bytes from %s", stotal, argv[2]);
    fclose(f);

    /* device buffers with guard bands; an empty shard passes NULL */
    size_t off = 0;
    for (int64_t k = 0; k < nsrc; ++k) {
        if (!sbytes[k]) continue;
        HIPCHECK(hipMalloc((void **)&sraw[k], sbytes[k] + 2 * GUARD));
        HIPCHECK(hipMemset(sraw[k], 0x5A, sbytes[k] + 2 * GUARD));
        HIPCHECK(hipMemcpy(sraw[k] + GUARD, sall + off, sbytes[k], hipMemcpyHostToDevice));
        sp[k] = sraw[k] + GUARD;
        off += sbytes[k];
    }
    for (int64_t k = 0; k < ndst; ++k) {
        if (!dbytes[k]) continue;
        HIPCHECK(hipMalloc((void **)&draw[k], dbytes[k] + 2 * GUARD));
        HIPCHECK(hipMemset(draw[k], 0x5A, dbytes[k] + 2 * GUARD));
        HIPCHECK(hipMemset(draw[k] + GUARD, 0xA5, dbytes[k]));
        dp[k] = draw[k] + GUARD;
    }

    hipStream_t stream = NULL;
    if (use_stream) HIPCHECK(hipStreamCreate(&stream));
    if (upload) RSCHECK(reshard_plan_upload(plan));
    for (int r = 0; r < repeat; ++r) RSCHECK(reshard_execute(plan, sp, dp, stream));
    HIPCHECK(hipStreamSynchronize(stream));
    HIPCHECK(hipGetLastError());

    /* guards untouched, sources unmodified, destinations out */
    off = 0;
    for (int64_t k = 0; k < nsrc; ++k) {
        if (!sbytes[k]) continue;
        HIPCHECK(hipMemcpy(host, sraw[k], sbytes[k] + 2 * GUARD, hipMemcpyDeviceToHost));
        for (size_t i = 0; i < GUARD; ++i)
            if (host[i] != 0x5A || host[GUARD + sbytes[k] + i] != 0x5A) FAIL("source %ld guard changed", (long)k);
        if (memcmp(host + GUARD, sall + off, sbytes[k])) FAIL("source %ld changed", (long)k);
        off += sbytes[k];
    }
    off = 0;
    for (int64_t k = 0; k < ndst; ++k) {
        if (!dbytes[k]) continue;
        HIPCHECK(hipMemcpy(host, draw[k], dbytes[k] + 2 * GUARD, hipMemcpyDeviceToHost));
        for (size_t i = 0; i < GUARD; ++i)
            if (host[i] != 0x5A || host[GUARD + dbytes[k] + i] != 0x5A) FAIL("destination %ld guard changed", (long)k);
        memcpy(dall + off, host + GUARD, dbytes[k]);
        off += dbytes[k];
    }
    f = fopen(argv[3], "wb");
    if (!f || fwrite(dall, 1, dtotal, f) != dtotal) FAIL("cannot write %s", argv[3]);
    fclose(f);

    if (use_stream) HIPCHECK(hipStreamDestroy(stream));
    for (int64_t k = 0; k < nsrc; ++k)
        if (sraw[k]) HIPCHECK(hipFree(sraw[k]));
    for (int64_t k = 0; k < ndst; ++k)
        if (draw[k]) HIPCHECK(hipFree(draw[k]));
    reshard_plan_destroy(plan);
    free(host), free(sall), free(dall), free(sbytes), free(dbytes), free(sraw), free(draw), free(sp), free(dp);
    printf("ok\n");
    return 0;
}
