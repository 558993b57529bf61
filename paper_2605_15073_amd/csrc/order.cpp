// Receiver order of the message-passing passes (cgtp_receiver_order), computed on the host.
//
// The receiver passes run their blocks in the order of recv_block (internal.h): slice by
// slice, and inside a slice each XCD takes a contiguous span of the receiver sequence. The
// sum over a receiver's CSR row does not depend on that sequence, so any permutation gives
// the same outputs bit for bit; a sequence in which neighbours in space are close together
// lets the receivers one XCD runs at once share their senders, whose fields then stay in
// that XCD's L2.
//
// Atom positions are not an input of the library, so they are rebuilt from the graph: a
// breadth-first spanning tree of each connected component places a node at its parent's
// position plus the edge vector of the tree edge. With unit directions every hop counts one
// unit, which distorts distances but keeps nearby atoms nearby; with displacement vectors
// the positions are the atoms' own (up to periodic images). Nodes are sorted by component,
// then by the Hilbert index of their position in the component's bounding box.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <vector>

#include "internal.h"

namespace {

constexpr int kHilbertBits = 10;  // per axis: 2^30 cells

// Hilbert index of the cell (X[0], X[1], X[2]) of a 2^b grid per axis: Skilling's
// transform of the axes to the transposed index, then its bits interleaved, most significant
// first (J. Skilling, "Programming the Hilbert curve", AIP Conf. Proc. 707 (2004) 381).
uint64_t hilbert3(uint32_t X[3], int b)
{
    const uint32_t top = 1u << (b - 1);
    for (uint32_t q = top; q > 1; q >>= 1) {
        const uint32_t low = q - 1;
        for (int i = 0; i < 3; ++i) {
            if (X[i] & q) {
                X[0] ^= low;  // invert the low bits of the first axis
            } else {          // exchange the low bits of the first axis and axis i
                const uint32_t t = (X[0] ^ X[i]) & low;
                X[0] ^= t;
                X[i] ^= t;
            }
        }
    }
    for (int i = 1; i < 3; ++i) X[i] ^= X[i - 1];  // Gray encoding
    uint32_t t = 0;
    for (uint32_t q = top; q > 1; q >>= 1)
        if (X[2] & q) t ^= q - 1;
    for (int i = 0; i < 3; ++i) X[i] ^= t;
    uint64_t h = 0;
    for (int bit = b - 1; bit >= 0; --bit)
        for (int i = 0; i < 3; ++i) h = (h << 1) | ((X[i] >> bit) & 1u);
    return h;
}

int check_csr(int64_t n, int64_t E, const int32_t *row_ptr, const int32_t *col)
{
    if (row_ptr[0] != 0 || row_ptr[n] != E)
        return cgtp::report(CGTP_ERR_CSR, "row_ptr[0] = %d and row_ptr[n] = %d, expected 0 and %lld",
                            row_ptr[0], row_ptr[n], (long long)E);
    for (int64_t i = 0; i < n; ++i)
        if (row_ptr[i + 1] < row_ptr[i])
            return cgtp::report(CGTP_ERR_CSR, "row_ptr decreases at row %lld", (long long)i);
    for (int64_t e = 0; e < E; ++e)
        if (col[e] < 0 || col[e] >= n)
            return cgtp::report(CGTP_ERR_CSR, "col[%lld] = %d is not a node", (long long)e, col[e]);
    return CGTP_OK;
}

}  // namespace

extern "C" int cgtp_receiver_order(int64_t n_nodes, int64_t n_edges, const int32_t *row_ptr,
                                   const int32_t *col, const float *edge_vec, int32_t *order)
{
    cgtp::clear_error();
    if (n_nodes < 0 || n_edges < 0) return cgtp::report(CGTP_ERR_ARG, "negative size");
    if (n_nodes >= 0x7fffffffLL || n_edges >= 0x7fffffffLL)
        return cgtp::report(CGTP_ERR_ARG, "sizes must be below 2^31 - 1");
    if (n_nodes == 0) return n_edges == 0 ? CGTP_OK : cgtp::report(CGTP_ERR_ARG, "edges without nodes");
    if (!row_ptr || !order || (n_edges > 0 && !col)) return cgtp::report(CGTP_ERR_ARG, "NULL argument");
    int st = check_csr(n_nodes, n_edges, row_ptr, col);
    if (st) return st;
    const int64_t n = n_nodes;
    // breadth-first discovery, component by component from the lowest unvisited node
    std::vector<int32_t> seq;
    seq.reserve((size_t)n);
    std::vector<int32_t> comp((size_t)n, -1);
    std::vector<double> pos(edge_vec ? 3 * (size_t)n : 0, 0.0);
    std::vector<int64_t> comp_start;
    int32_t ncomp = 0;
    for (int64_t root = 0; root < n; ++root) {
        if (comp[root] >= 0) continue;
        comp_start.push_back((int64_t)seq.size());
        comp[root] = ncomp;
        seq.push_back((int32_t)root);
        for (size_t h = seq.size() - 1; h < seq.size(); ++h) {
            const int32_t i = seq[h];
            for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
                const int32_t j = col[e];
                if (comp[j] >= 0) continue;
                comp[j] = ncomp;
                if (edge_vec)
                    for (int a = 0; a < 3; ++a)
                        pos[3 * (size_t)j + a] = pos[3 * (size_t)i + a] + (double)edge_vec[3 * (int64_t)e + a];
                seq.push_back(j);
            }
        }
        ++ncomp;
    }
    comp_start.push_back(n);
    if (!edge_vec) {
        std::copy(seq.begin(), seq.end(), order);
        return CGTP_OK;
    }
    // per component: the Hilbert index of each node's cell in the component's bounding box
    std::vector<std::pair<uint64_t, int32_t>> key;
    int64_t out = 0;
    for (int32_t c = 0; c < ncomp; ++c) {
        const int64_t a0 = comp_start[c], a1 = comp_start[c + 1];
        double lo[3], hi[3];
        for (int a = 0; a < 3; ++a) lo[a] = hi[a] = pos[3 * (size_t)seq[a0] + a];
        bool finite = true;
        for (int64_t h = a0; h < a1; ++h)
            for (int a = 0; a < 3; ++a) {
                const double x = pos[3 * (size_t)seq[h] + a];
                finite = finite && std::isfinite(x);
                lo[a] = std::min(lo[a], x);
                hi[a] = std::max(hi[a], x);
            }
        double ext = 0;
        for (int a = 0; a < 3; ++a) ext = std::max(ext, hi[a] - lo[a]);
        key.clear();
        const double cells = (double)(1u << kHilbertBits);
        for (int64_t h = a0; h < a1; ++h) {
            uint32_t X[3] = {0, 0, 0};
            if (finite && ext > 0)
                for (int a = 0; a < 3; ++a) {
                    const double f = (pos[3 * (size_t)seq[h] + a] - lo[a]) / ext * cells;
                    X[a] = (uint32_t)std::min(cells - 1, std::max(0.0, std::floor(f)));
                }
            key.emplace_back(hilbert3(X, kHilbertBits), seq[h]);
        }
        // ties (one cell) keep the breadth-first order
        std::stable_sort(key.begin(), key.end(),
                         [](const std::pair<uint64_t, int32_t> &x,
                            const std::pair<uint64_t, int32_t> &y) { return x.first < y.first; });
        for (const auto &k : key) order[out++] = k.second;
    }
    return CGTP_OK;
}
