/* A plain C user of libtopkv.so (no Python, no torch): one layer of a small
 * paged pool is packed (gather into the wire order [plane][token][head][dim]),
 * unpacked into a pool with another page size, packed again and compared; the
 * destination pool is then re-blocked back pool-to-pool and two head halves
 * are packed and checked against the full-head packed layer; the layer
 * engine packs both layers in one call and is checked against the per-layer
 * packs.  Then a
 * fixed-state layer: two requests' states are packed from a state cache and
 * unpacked into other slots of a second cache; and the device CRC-64 of
 * "123456789" is checked against the published CRC-64/XZ check value.
 *
 * Build:  gcc -std=c11 -D__HIP_PLATFORM_AMD__ -I/opt/rocm/include -Iinclude \
 *             paper_2607_28633_amd/examples/roundtrip.c \
 *             -Lpaper_2607_28633_amd -ltopkv -L/opt/rocm/lib -lamdhip64 -o roundtrip
 * Run:    LD_LIBRARY_PATH=paper_2607_28633_amd:/opt/rocm/lib ./roundtrip
 * Prints "roundtrip ok" and exits 0, or names the failing step and exits 1.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "topkv.h"

#define LAYERS 2
#define PLANES 2
#define HEADS 4
#define DIM 64
#define P_SRC 16
#define P_DST 5
#define PAGES 64
#define TOKENS 300

#define HIP_OK(x) do { if ((x) != hipSuccess) { fprintf(stderr, "HIP call failed: %s\n", #x); return 1; } } while (0)
#define TOPKV_OK_OR_FAIL(x) do { topkv_status_t st_ = (x); if (st_ != TOPKV_OK) { \
    fprintf(stderr, "%s: %s\n", #x, topkv_status_string(st_)); return 1; } } while (0)

/* A permutation of the pool's pages (a fragmented pool): page i of the
 * request lives at physical page (i * 37 + 11) mod PAGES. */
static void fill_table(int32_t* bt, int n_pages) {
    for (int i = 0; i < n_pages; ++i) bt[i] = (int32_t)((i * 37 + 11) % PAGES);
}

int main(void) {
    const size_t row = (size_t)HEADS * DIM * 2;
    const size_t pool_elems = (size_t)LAYERS * PAGES * PLANES * P_SRC * HEADS * DIM;
    const size_t dst_elems = (size_t)LAYERS * PAGES * PLANES * P_DST * HEADS * DIM;
    const size_t packed_bytes = (size_t)PLANES * TOKENS * row;
    const int layer = 1;
    const int pages_src = (TOKENS + P_SRC - 1) / P_SRC, pages_dst = (TOKENS + P_DST - 1) / P_DST;

    uint16_t* host_pool = malloc(pool_elems * 2);
    uint16_t* a = malloc(packed_bytes);
    uint16_t* b = malloc(packed_bytes);
    int32_t bt_src[PAGES], bt_dst[PAGES];
    if (!host_pool || !a || !b) return 1;
    for (size_t i = 0; i < pool_elems; ++i) host_pool[i] = (uint16_t)(i * 2654435761u >> 7);
    for (int i = 0; i < PAGES; ++i) bt_src[i] = bt_dst[i] = -1;      /* entries past the request: unused */
    fill_table(bt_src, pages_src);
    for (int i = 0; i < pages_dst; ++i) bt_dst[i] = (int32_t)((i * 13 + 5) % PAGES);

    void *d_pool, *d_dst, *d_back, *d_a, *d_b, *d_half, *d_bt_src, *d_bt_dst, *d_len;
    HIP_OK(hipMalloc(&d_pool, pool_elems * 2));
    HIP_OK(hipMalloc(&d_dst, dst_elems * 2));
    HIP_OK(hipMalloc(&d_back, pool_elems * 2));
    HIP_OK(hipMalloc(&d_a, packed_bytes));
    HIP_OK(hipMalloc(&d_b, packed_bytes));
    HIP_OK(hipMalloc(&d_half, packed_bytes));
    HIP_OK(hipMalloc(&d_bt_src, sizeof bt_src));
    HIP_OK(hipMalloc(&d_bt_dst, sizeof bt_dst));
    HIP_OK(hipMalloc(&d_len, sizeof(int32_t)));
    const int32_t len = TOKENS;
    HIP_OK(hipMemcpy(d_pool, host_pool, pool_elems * 2, hipMemcpyHostToDevice));
    HIP_OK(hipMemset(d_dst, 0, dst_elems * 2));
    HIP_OK(hipMemset(d_back, 0, pool_elems * 2));
    HIP_OK(hipMemcpy(d_bt_src, bt_src, sizeof bt_src, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(d_bt_dst, bt_dst, sizeof bt_dst, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(d_len, &len, sizeof len, hipMemcpyHostToDevice));

    topkv_pool_t src = {d_pool, PAGES, LAYERS, P_SRC, PLANES, HEADS, DIM, 2};
    topkv_pool_t dst = {d_dst, PAGES, LAYERS, P_DST, PLANES, HEADS, DIM, 2};
    topkv_pool_t back = {d_back, PAGES, LAYERS, P_SRC, PLANES, HEADS, DIM, 2};

    /* pack, unpack into page size 5, pack again */
    TOPKV_OK_OR_FAIL(topkv_pack_layer(&src, layer, d_bt_src, TOKENS, d_a, 0));
    TOPKV_OK_OR_FAIL(topkv_unpack_layer(d_a, &dst, layer, d_bt_dst, TOKENS, 0));
    TOPKV_OK_OR_FAIL(topkv_pack_layer(&dst, layer, d_bt_dst, TOKENS, d_b, 0));
    HIP_OK(hipDeviceSynchronize());
    HIP_OK(hipMemcpy(a, d_a, packed_bytes, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(b, d_b, packed_bytes, hipMemcpyDeviceToHost));
    if (memcmp(a, b, packed_bytes) != 0) { fprintf(stderr, "round trip through page size 5 differs\n"); return 1; }

    /* the wire order: token t of plane c starts row (c * TOKENS + t) of the packed layer */
    for (int c = 0; c < PLANES; ++c)
        for (int t = 0; t < TOKENS; t += 37) {
            const size_t page = (size_t)bt_src[t / P_SRC], slot = (size_t)(t % P_SRC);
            const uint16_t* want = host_pool + ((((size_t)layer * PAGES + page) * PLANES + c) * P_SRC + slot) * HEADS * DIM;
            if (memcmp(a + ((size_t)c * TOKENS + t) * HEADS * DIM, want, row) != 0) {
                fprintf(stderr, "packed row of plane %d token %d is not the pool's row\n", c, t);
                return 1;
            }
        }

    /* pool-to-pool re-block back to page size 16, then pack: the same layer */
    TOPKV_OK_OR_FAIL(topkv_reblock_layer(&dst, layer, d_bt_dst, PAGES, &back, layer, d_bt_src, PAGES, 1, d_len, 0));
    TOPKV_OK_OR_FAIL(topkv_pack_layer(&back, layer, d_bt_src, TOKENS, d_b, 0));
    HIP_OK(hipDeviceSynchronize());
    HIP_OK(hipMemcpy(b, d_b, packed_bytes, hipMemcpyDeviceToHost));
    if (memcmp(a, b, packed_bytes) != 0) { fprintf(stderr, "pool-to-pool re-block differs\n"); return 1; }

    /* head halves [0, 2) and [2, 4): side by side they are the full rows */
    const size_t half_bytes = packed_bytes / 2, half_row = row / 2;
    for (int h = 0; h < 2; ++h) {
        TOPKV_OK_OR_FAIL(topkv_pack_layer_heads(&src, layer, 1, d_bt_src, PAGES, d_len, 2 * h, 2, d_half,
                                                (int64_t)half_bytes, 0));
        HIP_OK(hipDeviceSynchronize());
        HIP_OK(hipMemcpy(b, d_half, half_bytes, hipMemcpyDeviceToHost));
        for (size_t r = 0; r < (size_t)PLANES * TOKENS; ++r)
            if (memcmp((const char*)b + r * half_row, (const char*)a + r * row + h * half_row, half_row) != 0) {
                fprintf(stderr, "head half %d differs at row %zu\n", h, r);
                return 1;
            }
    }

    /* the layer engine: both layers in one call per direction, layer z's packed block at z * packed_bytes;
     * block 1 is the layer packed above, block 0 the same as a single-layer pack of layer 0 */
    void* d_two;
    uint16_t* two = malloc(2 * packed_bytes);
    if (!two) return 1;
    HIP_OK(hipMalloc(&d_two, 2 * packed_bytes));
    TOPKV_OK_OR_FAIL(topkv_engine_pack_layers(&src, 0, LAYERS, 1, d_bt_src, PAGES, d_len, d_two,
                                              (int64_t)packed_bytes, (int64_t)(2 * packed_bytes), NULL, 0));
    TOPKV_OK_OR_FAIL(topkv_pack_layer(&src, 0, d_bt_src, TOKENS, d_b, 0));
    HIP_OK(hipDeviceSynchronize());
    HIP_OK(hipMemcpy(two, d_two, 2 * packed_bytes, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(b, d_b, packed_bytes, hipMemcpyDeviceToHost));
    if (memcmp((const char*)two + packed_bytes, a, packed_bytes) != 0 || memcmp(two, b, packed_bytes) != 0) {
        fprintf(stderr, "layer engine blocks differ from the per-layer packs\n");
        return 1;
    }
    hipFree(d_two);
    free(two);

    /* fixed-state layer: states of slots {3, 1} of layer 1, unpacked into slots {0, 2} of a second cache */
    enum { SLOTS = 4, STATE = 1000 };
    const size_t cache_bytes = (size_t)LAYERS * SLOTS * STATE;
    unsigned char* hc = malloc(cache_bytes);
    unsigned char* hs = malloc(cache_bytes);
    if (!hc || !hs) return 1;
    for (size_t i = 0; i < cache_bytes; ++i) hc[i] = (unsigned char)(i * 131u + 7u);
    void *d_cache, *d_cache2, *d_states, *d_slots, *d_slots2;
    HIP_OK(hipMalloc(&d_cache, cache_bytes));
    HIP_OK(hipMalloc(&d_cache2, cache_bytes));
    HIP_OK(hipMalloc(&d_states, 2 * STATE));
    HIP_OK(hipMalloc(&d_slots, 2 * sizeof(int32_t)));
    HIP_OK(hipMalloc(&d_slots2, 2 * sizeof(int32_t)));
    const int32_t slots[2] = {3, 1}, slots2[2] = {0, 2};
    HIP_OK(hipMemcpy(d_cache, hc, cache_bytes, hipMemcpyHostToDevice));
    HIP_OK(hipMemset(d_cache2, 0, cache_bytes));
    HIP_OK(hipMemcpy(d_slots, slots, sizeof slots, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(d_slots2, slots2, sizeof slots2, hipMemcpyHostToDevice));
    topkv_state_pool_t cache = {d_cache, SLOTS, STATE, LAYERS, 0};
    topkv_state_pool_t cache2 = {d_cache2, SLOTS, STATE, LAYERS, 0};
    topkv_launch_t on_null = {0, 0, 0};
    if (topkv_packed_state_bytes(&cache, 2) != 2 * STATE) { fprintf(stderr, "packed state bytes\n"); return 1; }
    TOPKV_OK_OR_FAIL(topkv_pack_state_layer(&cache, layer, 2, d_slots, d_states, 2 * STATE, &on_null));
    TOPKV_OK_OR_FAIL(topkv_unpack_state_layer(d_states, 2 * STATE, &cache2, layer, 2, d_slots2, &on_null));
    HIP_OK(hipDeviceSynchronize());
    HIP_OK(hipMemcpy(hs, d_cache2, cache_bytes, hipMemcpyDeviceToHost));
    for (size_t i = 0; i < cache_bytes; ++i) {
        const size_t l = i / ((size_t)SLOTS * STATE), sl = i / STATE % SLOTS, e = i % STATE;
        unsigned char want = 0;
        if (l == (size_t)layer && (sl == 0 || sl == 2))
            want = hc[((size_t)layer * SLOTS + (size_t)slots[sl / 2]) * STATE + e];
        if (hs[i] != want) { fprintf(stderr, "state cache byte %zu differs\n", i); return 1; }
    }

    /* CRC-64/XZ of "123456789" on the device: the published check value */
    const char msg[] = "123456789";
    void *d_msg, *d_ws, *d_crc;
    const int64_t ws_bytes = topkv_crc64_workspace_bytes(9);
    HIP_OK(hipMalloc(&d_msg, 16));
    HIP_OK(hipMalloc(&d_ws, (size_t)ws_bytes));
    HIP_OK(hipMalloc(&d_crc, sizeof(uint64_t)));
    HIP_OK(hipMemcpy(d_msg, msg, 9, hipMemcpyHostToDevice));
    TOPKV_OK_OR_FAIL(topkv_crc64(d_msg, 9, d_ws, ws_bytes, (uint64_t*)d_crc, 0));
    uint64_t crc = 0;
    HIP_OK(hipMemcpy(&crc, d_crc, sizeof crc, hipMemcpyDeviceToHost));
    if (crc != 0x995DC9BBDF1939FAull) { fprintf(stderr, "crc64 %016llx\n", (unsigned long long)crc); return 1; }

    hipFree(d_pool); hipFree(d_dst); hipFree(d_back); hipFree(d_a); hipFree(d_b); hipFree(d_half);
    hipFree(d_bt_src); hipFree(d_bt_dst); hipFree(d_len);
    hipFree(d_cache); hipFree(d_cache2); hipFree(d_states); hipFree(d_slots); hipFree(d_slots2);
    hipFree(d_msg); hipFree(d_ws); hipFree(d_crc);
    free(host_pool); free(a); free(b); free(hc); free(hs);
    printf("roundtrip ok\n");
    return 0;
}
