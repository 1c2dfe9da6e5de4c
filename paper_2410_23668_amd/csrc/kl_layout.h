// The packed weight layout: tile geometry, the arena's geometry for a model
// on a grid of nwg workgroups, the row maps, the body of the packing kernel
// (one 16-byte chunk of a packed matrix) and the list of packing jobs of a
// layer and of the classifier.  Shared by the host runtime, which runs the
// jobs with the packing kernel, and by the CPU round-trip test of the layout
// (compiled there with KL_HD defined empty).
//
// Packed matrices are 1 KiB tiles of 8 rows x 64 columns (bf16, row-major
// inside the tile); the tiles of one 8-row group are contiguous along K.  K is
// padded to 64 and rows to 8 with zeros.  Row maps give, for each packed row,
// (source id << 28) | source row, or -1 for a zero row.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <algorithm>
#include <vector>

#include "kl.h"

#ifndef KL_HD
#define KL_HD __host__ __device__
#endif

namespace kl {

constexpr int kTileRows = 8;              // rows of one packed weight tile
constexpr int kTileK = 64;                // columns of one packed weight tile
constexpr int kTileBytes = kTileRows * kTileK * 2;   // 1 KiB: one 16-byte load per lane

// Packed row and first column of 16-byte chunk idx of a packed matrix with KT
// k-tiles per row group (lane l of a tile's 64 chunks holds row l / 8,
// columns 8 (l % 8) .. + 7).
KL_HD inline void pack_chunk_coords(size_t idx, int KT, int &prow, int &col) {
    const int lane = (int)(idx % 64);
    const size_t tile = idx / 64;
    const int kt = (int)(tile % (size_t)KT);
    const int rg = (int)(tile / (size_t)KT);
    prow = rg * kTileRows + lane / 8;
    col = kt * kTileK + (lane % 8) * 8;
}

// The 8 bf16 values of chunk idx, packed two per word: columns >= K and rows
// mapped to -1 are zero; src[s] + row ld is source s's row.
KL_HD inline void pack_chunk(size_t idx, int KT, int K, int ld, const int32_t *rowmap,
                             const uint16_t *const src[3], uint32_t w[4]) {
    int prow, col;
    pack_chunk_coords(idx, KT, prow, col);
    const int m = rowmap[prow];
    w[0] = w[1] = w[2] = w[3] = 0u;
    if (m < 0) return;
    const uint16_t *row = src[m >> 28] + (size_t)(m & 0x0fffffff) * ld;
    for (int e = 0; e < 8; ++e) {
        const uint32_t v = (col + e < K) ? row[col + e] : 0u;
        w[e >> 1] |= v << (16 * (e & 1));
    }
}

// Packed bias row r (fp32): the q/k/v bias of the source row the q/k/v row
// map gives r, zero for a padding row.
KL_HD inline float pack_bias_row(int r, const int32_t *rowmap, const uint16_t *const src[3]) {
    const int m = rowmap[r];
    if (m < 0) return 0.f;
    const uint32_t bits = (uint32_t)src[m >> 28][m & 0x0fffffff] << 16;
    float f;
    __builtin_memcpy(&f, &bits, 4);
    return f;
}

inline size_t layout_align(size_t v, size_t a) { return (v + a - 1) / a * a; }
inline int layout_pad_k(int v) { return (v + kTileK - 1) / kTileK * kTileK; }

// FFN column blocks: the number of blocks dividing the ffn k-tiles, at most
// 32 and at most the grid (the largest such).
inline int layout_ffn_blocks(int ktf, int nwg) {
    int best = 1;
    for (int s = 1; s <= std::min(32, std::min(ktf, nwg)); ++s)
        if (ktf % s == 0) best = s;
    return best;
}

struct Geometry {
    int nwg;
    int E, topk;               // experts per layer (1: the dense MLP), experts per token
    int Hp, Ap, Fp;            // K extents padded to kTileK: hidden, n_heads d, ffn
    int KTH, KTF, KTq;         // k-tiles of hidden, ffn, one head
    int Sg;                    // workgroups per KV head
    int Sc, Rc, KTc;           // FFN column blocks, workgroups per block, k-tiles per block
    int qkv_rg;                // row groups of one KV head's q/k/v block
    int o_rg, gu_rg, down_rg, head_rg;
    // arena: [layer 0 .. L-1][final norm][LM head][embedding][zero tile]
    size_t off_attn_norm, off_ffn_norm, off_qkv_bias, off_qkv, off_o, off_router, off_gu,
        off_down, layer_stride;
    size_t gu_estride, down_estride;   // bytes from one expert's gate/up (down) to the next
    size_t off_final_norm, off_lm_head, off_embed, off_dummy, arena_bytes;
};

// Per layer: the two norm gains (fp32, padded to Hp), the Q/K/V biases if
// the model has them (fp32, packed row order), the q/k/v matrix
// grouped per KV head (its G query heads, its key, its value; query and key
// rows in rotation pairs (i, i + d/2)), the O projection per query head (its
// d columns), with experts the router (one packed row group), then per
// expert (or once) gate/up with rows interleaved (gate i, up i) and the down
// projection per FFN column block.  With experts, each of the top_k expert
// slots of a token has nwg / top_k workgroups, so the FFN column blocks are
// counted against that.
inline Geometry layout_geometry(const kl_config &c, int nwg) {
    Geometry G{};
    const int d = c.head_dim, g = c.n_heads / c.n_kv_heads;
    G.nwg = nwg;
    G.E = c.n_experts > 1 ? c.n_experts : 1;
    G.topk = c.n_experts > 1 ? c.top_k : 1;
    G.Hp = layout_pad_k(c.hidden);
    G.Ap = layout_pad_k(c.n_heads * d);
    G.Fp = layout_pad_k(c.ffn_dim);
    G.KTH = G.Hp / kTileK;
    G.KTF = G.Fp / kTileK;
    G.KTq = d / kTileK;
    G.Sg = nwg / c.n_kv_heads;
    G.Sc = layout_ffn_blocks(G.KTF, nwg / G.topk);
    G.Rc = nwg / G.topk / G.Sc;
    G.KTc = G.KTF / G.Sc;
    G.qkv_rg = (g + 2) * d / kTileRows;
    G.o_rg = c.hidden / kTileRows;
    G.gu_rg = 2 * c.ffn_dim / kTileRows;
    G.down_rg = c.hidden / kTileRows;
    G.head_rg = (c.vocab + kTileRows - 1) / kTileRows;
    const size_t A = 4096;
    size_t off = 0;
    G.off_attn_norm = off; off = layout_align(off + (size_t)G.Hp * 4, A);
    G.off_ffn_norm = off;  off = layout_align(off + (size_t)G.Hp * 4, A);
    // Q/K/V biases (fp32, in the packed row order of the q/k/v matrix)
    G.off_qkv_bias = off;
    if (c.qkv_bias) off = layout_align(off + (size_t)c.n_kv_heads * G.qkv_rg * kTileRows * 4, A);
    G.off_qkv = off;
    off = layout_align(off + (size_t)c.n_kv_heads * G.qkv_rg * G.KTH * kTileBytes, A);
    G.off_o = off;
    off = layout_align(off + (size_t)c.n_heads * G.o_rg * G.KTq * kTileBytes, A);
    G.off_router = off;
    if (G.E > 1) off = layout_align(off + (size_t)G.KTH * kTileBytes, A);
    G.gu_estride = layout_align((size_t)G.gu_rg * G.KTH * kTileBytes, A);
    G.off_gu = off;        off += (size_t)G.E * G.gu_estride;
    G.down_estride = layout_align((size_t)G.Sc * G.down_rg * G.KTc * kTileBytes, A);
    G.off_down = off;      off += (size_t)G.E * G.down_estride;
    G.layer_stride = off;
    off = G.layer_stride * c.n_layers;
    G.off_final_norm = off; off = layout_align(off + (size_t)G.Hp * 4, A);
    G.off_lm_head = off;    off = layout_align(off + (size_t)G.head_rg * G.KTH * kTileBytes, A);
    G.off_embed = off;      off = layout_align(off + (size_t)c.vocab * c.hidden * 2, A);
    G.off_dummy = off;      off = layout_align(off + kTileBytes, A);
    G.arena_bytes = off;
    return G;
}

enum RowMap { kMapQkv = 0, kMapHidden = 1, kMapGateUp = 2, kMapHead = 3, kMapRouter = 4 };

inline std::vector<int32_t> row_map(const kl_config &c, RowMap which) {
    std::vector<int32_t> m;
    if (which == kMapQkv) {
        const int d = c.head_dim, half = d / 2, G = c.n_heads / c.n_kv_heads;
        const auto pair = [&](int j) { return j / 2 + (j % 2) * half; };
        for (int g = 0; g < c.n_kv_heads; ++g) {
            for (int h = g * G; h < (g + 1) * G; ++h)
                for (int j = 0; j < d; ++j) m.push_back((0 << 28) | (h * d + pair(j)));
            for (int j = 0; j < d; ++j) m.push_back((1 << 28) | (g * d + pair(j)));
            for (int j = 0; j < d; ++j) m.push_back((2 << 28) | (g * d + j));
        }
    } else if (which == kMapHidden) {
        for (int r = 0; r < c.hidden; ++r) m.push_back(r);
    } else if (which == kMapGateUp) {
        for (int i = 0; i < c.ffn_dim; ++i) {
            m.push_back(i);                 // gate row i
            m.push_back((1 << 28) | i);     // up row i
        }
    } else if (which == kMapHead) {
        const int rows = (c.vocab + kTileRows - 1) / kTileRows * kTileRows;
        for (int r = 0; r < rows; ++r) m.push_back(r < c.vocab ? r : -1);
    } else {   // the router: one row group of n_experts rows
        for (int r = 0; r < kTileRows; ++r) m.push_back(r < c.n_experts ? r : -1);
    }
    return m;
}

// The caller's source matrices (nn.Linear layout [out][in], bf16).
enum Source { kSrcNone = -1, kSrcWq, kSrcWk, kSrcWv, kSrcWo, kSrcGate, kSrcUp, kSrcDown,
              kSrcLmHead, kSrcRouter };

// One run of the packing kernel: n_rg row groups x KT k-tiles at byte
// offset dst (of the layer, or of the arena for the classifier), from the K
// columns starting at element col0 of rows with stride ld of the sources.
struct PackJob {
    size_t dst;
    int n_rg, KT, K, ld;
    RowMap map;
    Source src[3];
    size_t col0;
};

inline std::vector<PackJob> layer_pack_jobs(const kl_config &c, const Geometry &G) {
    std::vector<PackJob> jobs;
    const int d = c.head_dim;
    jobs.push_back({G.off_qkv, c.n_kv_heads * G.qkv_rg, G.KTH, c.hidden, c.hidden, kMapQkv,
                    {kSrcWq, kSrcWk, kSrcWv}, 0});
    for (int h = 0; h < c.n_heads; ++h)   // Wo[:, query head h]
        jobs.push_back({G.off_o + (size_t)h * G.o_rg * G.KTq * kTileBytes, G.o_rg, G.KTq, d,
                        c.n_heads * d, kMapHidden, {kSrcWo, kSrcNone, kSrcNone}, (size_t)h * d});
    if (G.E > 1)   // the router [E][H]
        jobs.push_back({G.off_router, 1, G.KTH, c.hidden, c.hidden, kMapRouter,
                        {kSrcRouter, kSrcNone, kSrcNone}, 0});
    for (int e = 0; e < G.E; ++e) {   // (expert e's matrices: source offsets e F H)
        const size_t eo = (size_t)e * c.ffn_dim * c.hidden;
        jobs.push_back({G.off_gu + e * G.gu_estride, G.gu_rg, G.KTH, c.hidden, c.hidden,
                        kMapGateUp, {kSrcGate, kSrcUp, kSrcNone}, eo});
        for (int j = 0; j < G.Sc; ++j) {   // Wd[:, column block j]
            const int c0 = j * G.KTc * kTileK;
            jobs.push_back({G.off_down + e * G.down_estride +
                                (size_t)j * G.down_rg * G.KTc * kTileBytes,
                            G.down_rg, G.KTc,
                            std::max(0, std::min(c.ffn_dim - c0, G.KTc * kTileK)), c.ffn_dim,
                            kMapHidden, {kSrcDown, kSrcNone, kSrcNone}, eo + (size_t)c0});
        }
    }
    return jobs;
}

inline PackJob head_pack_job(const kl_config &c, const Geometry &G) {
    return {G.off_lm_head, G.head_rg, G.KTH, c.hidden, c.hidden, kMapHead,
            {kSrcLmHead, kSrcNone, kSrcNone}, 0};
}

}  // namespace kl
