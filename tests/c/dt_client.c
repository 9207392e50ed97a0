/*
 * A C11 client of libdtree that includes nothing but <dtree.h> and the C library: the
 * tests build it with gcc (-std=c11 -pedantic -Werror) to show that the header is plain C
 * and that a C program, with no HIP code and no Python, can use the library.
 *
 *   dt_client check TREE                   host only: dt_abi_version and dt_tree_check
 *   dt_client classify TREE RECORDS OUT ALGO
 *                                          dt_tree_create, then dt_classify_host (records
 *                                          and labels in host memory), ALGO 0 data,
 *                                          1 speculative, 2 path
 *   dt_client forest FOREST RECORDS OUT ALGO
 *                                          dt_forest_create, then dt_forest_classify_host
 *
 * TREE:    int32 n_nodes, n_features, n_classes, then n_nodes dt_node records
 * FOREST:  int32 n_trees, n_features, n_classes, then n_trees + 1 int32 tree offsets,
 *          then the dt_node records of every tree
 * RECORDS: int64 n, then n rows of n_features floats
 * OUT:     n int32 class labels
 * "check" prints one line "depth windows levels" of the tree's data encoding.  Any
 * library error prints the status and dt_last_error() and exits with the status code.
 */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "dtree.h"

static void *read_all(const char *path, long *size) {
    FILE *f = fopen(path, "rb");
    if (!f) {
        perror(path);
        exit(100);
    }
    fseek(f, 0, SEEK_END);
    *size = ftell(f);
    fseek(f, 0, SEEK_SET);
    void *buf = malloc(*size > 0 ? (size_t)*size : 1);
    if (!buf || fread(buf, 1, (size_t)*size, f) != (size_t)*size) {
        fprintf(stderr, "%s: read failed\n", path);
        exit(100);
    }
    fclose(f);
    return buf;
}

static void check(dt_status st, const char *what) {
    if (st != DT_OK) {
        fprintf(stderr, "%s: %s (%s)\n", what, dt_status_string(st), dt_last_error());
        exit((int)st);
    }
}

/* Records file: n rows of n_features floats after an int64 count. */
static const float *records(const char *path, int32_t n_features, int64_t *n) {
    long size;
    const char *buf = read_all(path, &size);
    memcpy(n, buf, sizeof *n);
    if (size != (long)(8 + *n * n_features * 4)) {
        fprintf(stderr, "%s: size does not match %lld rows\n", path, (long long)*n);
        exit(100);
    }
    return (const float *)(buf + 8);
}

static void write_labels(const char *path, const int32_t *labels, int64_t n) {
    FILE *f = fopen(path, "wb");
    if (!f || fwrite(labels, 4, (size_t)n, f) != (size_t)n) {
        fprintf(stderr, "%s: write failed\n", path);
        exit(100);
    }
    fclose(f);
}

int main(int argc, char **argv) {
    if (argc < 3) {
        fprintf(stderr, "usage: dt_client check|classify|forest FILE [RECORDS OUT ALGO]\n");
        return 100;
    }
    if (dt_abi_version() != DT_ABI_VERSION) {
        fprintf(stderr, "library ABI %d, header ABI %d\n", (int)dt_abi_version(),
                DT_ABI_VERSION);
        return 101;
    }
    long size;
    const char *buf = read_all(argv[2], &size);
    int32_t head[3];
    memcpy(head, buf, sizeof head);
    const int32_t n_features = head[1], n_classes = head[2];
    const int forest = strcmp(argv[1], "forest") == 0;
    const int32_t n_trees = forest ? head[0] : 1;
    const int32_t *offsets = (const int32_t *)(buf + 12);
    const int32_t n_nodes = forest ? offsets[n_trees] : head[0];
    const dt_node *nodes =
        (const dt_node *)(buf + 12 + (forest ? 4 * (long)(n_trees + 1) : 0));

    if (strcmp(argv[1], "check") == 0) {
        dt_tree_info info;
        check(dt_tree_check(nodes, n_nodes, n_features, n_classes, NULL, &info),
              "dt_tree_check");
        printf("%d %d %d\n", (int)info.data_window_depth, (int)info.data_windows,
               (int)info.data_levels);
        return 0;
    }
    if (argc < 6) {
        fprintf(stderr, "classify and forest need RECORDS OUT ALGO\n");
        return 100;
    }
    int64_t n;
    const float *x = records(argv[3], n_features, &n);
    int32_t *labels = malloc(n > 0 ? (size_t)n * 4 : 4);
    const dt_algo algo = (dt_algo)atoi(argv[5]);
    dt_pipeline *pipe = NULL;
    check(dt_pipeline_create(n_features, NULL, &pipe), "dt_pipeline_create");
    if (forest) {
        dt_forest *f = NULL;
        check(dt_forest_create(nodes, offsets, n_trees, n_features, n_classes, NULL, &f),
              "dt_forest_create");
        check(dt_forest_classify_host(f, pipe, x, n, n_features, labels, DT_OUT_CLASS_I32,
                                      algo, NULL),
              "dt_forest_classify_host");
        dt_forest_destroy(f);
    } else {
        dt_tree *t = NULL;
        check(dt_tree_create(nodes, n_nodes, n_features, n_classes, NULL, &t),
              "dt_tree_create");
        check(dt_classify_host(t, pipe, x, n, n_features, labels, DT_OUT_CLASS_I32, algo,
                               NULL),
              "dt_classify_host");
        dt_tree_destroy(t);
    }
    dt_pipeline_destroy(pipe);
    write_labels(argv[4], labels, n);
    free(labels);
    return 0;
}
