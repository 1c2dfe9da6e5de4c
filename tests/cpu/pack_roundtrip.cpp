// Round trip of the packed weight layout on the host: seeded source matrices
// are packed with the library's own plan (layout_geometry, layer_pack_jobs,
// head_pack_job, row_map and pack_chunk, the body the packing kernel runs per
// 16-byte chunk), then every element of every packed matrix is read back the
// way the kernel's consumers interpret it, written here from the layout's
// description rather than from the row maps:
//   q/k/v, per KV head g, rows of its block: its G query heads, its key, its
//     value; inside a query or key head, packed rows 2i and 2i + 1 are dims i
//     and i + d/2 (the RoPE epilogue rotates them as a pair);
//   O projection, per query head h: rows are the output rows, columns h's d;
//   gate/up: packed row 2i is gate row i, 2i + 1 up row i;
//   down projection, per FFN column block j: columns j KTc 64 ..;
//   LM head: rows are vocabulary rows, padding rows zero;
//   Q/K/V biases (fp32): in the q/k/v matrix's packed row order;
//   with experts: the router (one row group of the experts' rows, zero
//   padded), and per expert e its own gate/up and down matrices at the
//   expert strides, read from the e-th stacked source matrix;
// and every column past a matrix's K is zero.  Also: the jobs' regions lie
// inside the layer (or the arena) and do not overlap.
// Prints "pack round trip OK" and exits 0, else prints the failures, exit 1.
#include <cstdint>
#include <cstdio>
#include <string>
#include <vector>

#include "kl_layout.h"

using namespace kl;

namespace {

int g_fail = 0;
void fail(const std::string &what) {
    if (g_fail < 20) std::fprintf(stderr, "FAIL: %s\n", what.c_str());
    ++g_fail;
}

uint64_t mix(uint64_t x) {   // SplitMix64 output function (any fixed hash will do)
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}

// a nonzero value per (matrix, row, column), so zeros can only be padding
uint16_t val(int m, int r, int k) {
    return (uint16_t)(1 + mix(((uint64_t)m << 48) ^ ((uint64_t)r << 24) ^ (uint64_t)k) % 65535);
}

// element (prow, col) of a packed matrix with KT k-tiles per row group
uint16_t packed_at(const std::vector<uint16_t> &arena, size_t base_bytes, int KT, int prow,
                   int col) {
    const size_t tile = (size_t)(prow / 8) * KT + col / 64;
    return arena[base_bytes / 2 + tile * 512 + (size_t)(prow % 8) * 64 + col % 64];
}

void run(const char *name, kl_config c, int nwg) {
    const Geometry G = layout_geometry(c, nwg);
    const int H = c.hidden, F = c.ffn_dim, V = c.vocab, d = c.head_dim;
    const int nq = c.n_heads, nkv = c.n_kv_heads, g = nq / nkv;
    // sources, nn.Linear layout [out][in]
    std::vector<std::vector<uint16_t>> src(9);
    const int E = c.n_experts > 1 ? c.n_experts : 1;
    auto fill = [&](int id, int rows, int cols) {
        src[id].resize((size_t)rows * cols);
        for (int r = 0; r < rows; ++r)
            for (int k = 0; k < cols; ++k) src[id][(size_t)r * cols + k] = val(id, r, k);
    };
    fill(kSrcWq, nq * d, H);
    fill(kSrcWk, nkv * d, H);
    fill(kSrcWv, nkv * d, H);
    fill(kSrcWo, H, nq * d);
    fill(kSrcGate, E * F, H);   // (experts stacked)
    fill(kSrcUp, E * F, H);
    fill(kSrcDown, E * H, F);
    fill(kSrcLmHead, V, H);
    if (E > 1) fill(kSrcRouter, E, H);
    // Q/K/V biases (ids 8..10, one row of nq d, nkv d, nkv d values)
    std::vector<std::vector<uint16_t>> bias(3);
    for (int k = 0; k < 3; ++k) {
        bias[k].resize((size_t)(k == 0 ? nq : nkv) * d);
        for (size_t i = 0; i < bias[k].size(); ++i) bias[k][i] = val(8 + k, 0, (int)i);
    }

    // pack layer 0 and the classifier into an arena, as the loader does
    std::vector<uint16_t> arena(G.arena_bytes / 2, 0);
    std::vector<std::pair<size_t, size_t>> regions;
    auto pack = [&](const PackJob &J, size_t base) {
        const std::vector<int32_t> map = row_map(c, J.map);
        const uint16_t *s[3];
        for (int k = 0; k < 3; ++k)
            s[k] = J.src[k] == kSrcNone ? nullptr : src[J.src[k]].data() + J.col0;
        if ((size_t)J.n_rg * kTileRows > map.size()) fail(std::string(name) + ": row map too short");
        const size_t chunks = (size_t)J.n_rg * J.KT * 64;
        for (size_t idx = 0; idx < chunks; ++idx) {
            uint32_t w[4];
            pack_chunk(idx, J.KT, J.K, J.ld, map.data(), s, w);
            for (int e = 0; e < 8; ++e)
                arena[(base + J.dst) / 2 + idx * 8 + e] = (uint16_t)(w[e >> 1] >> (16 * (e & 1)));
        }
        regions.push_back({base + J.dst, base + J.dst + chunks * 16});
    };
    for (const PackJob &J : layer_pack_jobs(c, G)) pack(J, 0);
    pack(head_pack_job(c, G), 0);
    // the bias vector, as the bias packing kernel writes it
    std::vector<float> packed_bias;
    if (c.qkv_bias) {
        const std::vector<int32_t> map = row_map(c, kMapQkv);
        const uint16_t *s[3] = {bias[0].data(), bias[1].data(), bias[2].data()};
        const int rows = nkv * G.qkv_rg * kTileRows;
        for (int r = 0; r < rows; ++r) packed_bias.push_back(pack_bias_row(r, map.data(), s));
        regions.push_back({G.off_qkv_bias, G.off_qkv_bias + (size_t)rows * 4});
    }

    // regions: inside their homes, no overlap
    for (size_t i = 0; i < regions.size(); ++i) {
        const bool in_layer = regions[i].second <= G.layer_stride;
        const bool is_head = regions[i].first == G.off_lm_head;
        if (!(in_layer || (is_head && regions[i].second <= G.off_embed)))
            fail(std::string(name) + ": a packed matrix leaves its region");
        for (size_t j = 0; j < i; ++j)
            if (regions[i].first < regions[j].second && regions[j].first < regions[i].second)
                fail(std::string(name) + ": two packed matrices overlap");
    }

    auto expect = [&](const char *what, uint16_t got, uint16_t want, int r, int k) {
        if (got != want)
            fail(std::string(name) + ": " + what + " row " + std::to_string(r) + " col " +
                 std::to_string(k) + ": " + std::to_string(got) + " != " + std::to_string(want));
    };
    // q/k/v
    const int hrows = (g + 2) * d;
    for (int kv = 0; kv < nkv; ++kv)
        for (int lr = 0; lr < hrows; ++lr)
            for (int k = 0; k < G.Hp; ++k) {
                const uint16_t got = packed_at(arena, G.off_qkv, G.KTH, kv * hrows + lr, k);
                uint16_t want = 0;
                if (k < H) {
                    if (lr < (g + 1) * d) {   // query or key head: pairs (i, i + d/2)
                        const int i = (lr % d) / 2, dim = (lr % 2 == 0) ? i : i + d / 2;
                        want = lr < g * d ? val(kSrcWq, (kv * g + lr / d) * d + dim, k)
                                          : val(kSrcWk, kv * d + dim, k);
                    } else {
                        want = val(kSrcWv, kv * d + (lr - (g + 1) * d), k);
                    }
                }
                expect("qkv", got, want, kv * hrows + lr, k);
            }
    // biases: packed row kv hrows + lr is the bias of the same source row as above
    if (c.qkv_bias)
        for (int kv = 0; kv < nkv; ++kv)
            for (int lr = 0; lr < hrows; ++lr) {
                uint16_t want;
                if (lr < (g + 1) * d) {
                    const int i = (lr % d) / 2, dim = (lr % 2 == 0) ? i : i + d / 2;
                    want = lr < g * d ? bias[0][(size_t)(kv * g + lr / d) * d + dim]
                                      : bias[1][(size_t)kv * d + dim];
                } else {
                    want = bias[2][(size_t)kv * d + (lr - (g + 1) * d)];
                }
                const float f = packed_bias[(size_t)kv * hrows + lr];
                uint32_t bits;
                __builtin_memcpy(&bits, &f, 4);
                if ((bits & 0xffffu) != 0 || (bits >> 16) != want)
                    fail(std::string(name) + ": bias row " + std::to_string(kv * hrows + lr));
            }
    // O projection per query head
    for (int h = 0; h < nq; ++h)
        for (int r = 0; r < H; ++r)
            for (int k = 0; k < d; ++k)
                expect("o", packed_at(arena, G.off_o + (size_t)h * G.o_rg * G.KTq * kTileBytes,
                                      G.KTq, r, k),
                       val(kSrcWo, r, h * d + k), r, k);
    // per expert: gate/up interleaved, down projection per FFN column block
    for (int e = 0; e < E; ++e) {
        for (int r = 0; r < 2 * F; ++r)
            for (int k = 0; k < G.Hp; ++k)
                expect("gate/up", packed_at(arena, G.off_gu + e * G.gu_estride, G.KTH, r, k),
                       k < H ? val(r % 2 == 0 ? kSrcGate : kSrcUp, e * F + r / 2, k) : 0, r, k);
        for (int j = 0; j < G.Sc; ++j)
            for (int r = 0; r < H; ++r)
                for (int k = 0; k < G.KTc * kTileK; ++k) {
                    const int col = j * G.KTc * kTileK + k;
                    expect("down",
                           packed_at(arena,
                                     G.off_down + e * G.down_estride +
                                         (size_t)j * G.down_rg * G.KTc * kTileBytes,
                                     G.KTc, r, k),
                           col < F ? val(kSrcDown, e * H + r, col) : 0, r, col);
                }
    }
    // the router: E rows, zero padding rows
    if (E > 1)
        for (int r = 0; r < kTileRows; ++r)
            for (int k = 0; k < G.Hp; ++k)
                expect("router", packed_at(arena, G.off_router, G.KTH, r, k),
                       (r < E && k < H) ? val(kSrcRouter, r, k) : 0, r, k);
    // LM head, padding rows zero
    for (int r = 0; r < G.head_rg * kTileRows; ++r)
        for (int k = 0; k < G.Hp; ++k)
            expect("lm head", packed_at(arena, G.off_lm_head, G.KTH, r, k),
                   (r < V && k < H) ? val(kSrcLmHead, r, k) : 0, r, k);
}

}  // namespace

int main() {
    //            L  H    nq nkv d    F    V    theta  eps    max_batch max_seq  qkv_bias
    run("d64 padded", {1, 136, 4, 2, 64, 200, 37, 1e4f, 1e-5f, 1, 64, 0}, 16);
    run("d64 group 8", {1, 128, 8, 1, 64, 96, 20, 1e4f, 1e-5f, 1, 64, 0}, 32);
    run("d128 group 4", {1, 256, 8, 2, 128, 320, 50, 5e5f, 1e-5f, 1, 64, 0}, 256);
    run("d128 group 1", {1, 192, 2, 2, 128, 136, 9, 5e5f, 1e-5f, 1, 64, 0}, 7);
    run("d128 group 3 bias", {1, 192, 6, 2, 128, 200, 11, 1e6f, 1e-6f, 1, 64, 1}, 24);
    run("d64 group 2 bias", {1, 136, 4, 2, 64, 200, 37, 1e4f, 1e-5f, 1, 64, 1}, 16);
    //                    L  H    nq nkv d    F    V   theta  eps  mb ms  bias E  k
    run("d128 experts 4 top 2", {1, 192, 4, 2, 128, 320, 11, 1e6f, 1e-5f, 1, 64, 0, 4, 2}, 16);
    run("d64 experts 8 top 1", {1, 136, 4, 2, 64, 200, 37, 1e4f, 1e-5f, 1, 64, 0, 8, 1}, 7);
    if (g_fail) {
        std::fprintf(stderr, "%d failures\n", g_fail);
        return 1;
    }
    std::printf("pack round trip OK\n");
    return 0;
}
