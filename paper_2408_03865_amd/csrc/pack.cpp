// pack.cpp -- host-side packing plans (§3.1, §5): which rows and offsets the
// variable-length sequences of a stream occupy, and the position indices that
// describe the result.  Plain C++, no device code.
#include <algorithm>
#include <cstdint>
#include <numeric>
#include <vector>

#include "packmamba.h"

namespace {

struct Plan {
    std::vector<packmamba_piece> pieces;
    int64_t rows = 0;
};

// In received order; a sequence that does not fit the rest of the current row seals
// it (the rest is padding).  A sequence longer than a row is truncated to a row.
void plan_sequential(const int64_t* len, int64_t n, int64_t L, Plan& p) {
    int64_t used = L;                  // no open row yet
    for (int64_t i = 0; i < n; ++i) {
        const int64_t m = std::min(len[i], L);
        if (used + m > L) { ++p.rows; used = 0; }
        p.pieces.push_back({i, p.rows - 1, used, m, 0});
        used += m;
    }
}

// Windows of `window` sequences, each sorted by length (longest first, ties in
// received order) and placed first-fit into the rows opened for that window; the
// window's rows are sealed when it ends.
void plan_greedy(const int64_t* len, int64_t n, int64_t L, int64_t window, Plan& p) {
    for (int64_t w0 = 0; w0 < n; w0 += window) {
        const int64_t w1 = std::min(n, w0 + window);
        std::vector<int64_t> idx(w1 - w0);
        std::iota(idx.begin(), idx.end(), w0);
        std::stable_sort(idx.begin(), idx.end(), [&](int64_t a, int64_t b) { return len[a] > len[b]; });
        std::vector<int64_t> used;      // fill of the rows opened in this window
        const int64_t base = p.rows;
        for (int64_t i : idx) {
            const int64_t m = std::min(len[i], L);
            size_t r = 0;
            while (r < used.size() && used[r] + m > L) ++r;
            if (r == used.size()) used.push_back(0);
            p.pieces.push_back({i, base + (int64_t)r, used[r], m, 0});
            used[r] += m;
        }
        p.rows += (int64_t)used.size();
    }
}

// In received order, every row filled to the end: a sequence that does not fit is
// cut at the row end and continues at the start of the next row (its position
// indices carry on), so only the last row holds padding.  Exact with the state
// passing of the operators.
void plan_cut(const int64_t* len, int64_t n, int64_t L, Plan& p) {
    int64_t used = L;
    for (int64_t i = 0; i < n; ++i) {
        int64_t done = 0;
        while (done < len[i]) {
            if (used == L) { ++p.rows; used = 0; }
            const int64_t m = std::min(len[i] - done, L - used);
            p.pieces.push_back({i, p.rows - 1, used, m, done});
            used += m;
            done += m;
        }
    }
}

}  // namespace

extern "C" {

int packmamba_pack_plan(const int64_t* lengths, int64_t count, int64_t seqlen, int32_t policy,
                        int64_t window, packmamba_piece* pieces, int64_t max_pieces,
                        int64_t* n_pieces, int64_t* n_rows) {
    if ((!lengths && count > 0) || !n_pieces || !n_rows) return PACKMAMBA_ERR_NULL;
    if (count < 0 || seqlen <= 0) return PACKMAMBA_ERR_SHAPE;
    for (int64_t i = 0; i < count; ++i)
        if (lengths[i] <= 0) return PACKMAMBA_ERR_SHAPE;
    Plan p;
    switch (policy) {
        case PACKMAMBA_PACK_SEQUENTIAL: plan_sequential(lengths, count, seqlen, p); break;
        case PACKMAMBA_PACK_GREEDY:
            if (window <= 0) return PACKMAMBA_ERR_SHAPE;
            plan_greedy(lengths, count, seqlen, window, p);
            break;
        case PACKMAMBA_PACK_CUT: plan_cut(lengths, count, seqlen, p); break;
        default: return PACKMAMBA_ERR_UNSUPPORTED;
    }
    *n_pieces = (int64_t)p.pieces.size();
    *n_rows = p.rows;
    if (!pieces) return PACKMAMBA_OK;                       // sizing query
    if ((int64_t)p.pieces.size() > max_pieces) return PACKMAMBA_ERR_WORKSPACE;
    std::copy(p.pieces.begin(), p.pieces.end(), pieces);
    return PACKMAMBA_OK;
}

int packmamba_pack_positions(const packmamba_piece* pieces, int64_t n_pieces, int64_t n_rows,
                             int64_t seqlen, int32_t* position_indices) {
    if ((!pieces && n_pieces > 0) || !position_indices) return PACKMAMBA_ERR_NULL;
    if (n_rows < 0 || seqlen <= 0 || seqlen > INT32_MAX) return PACKMAMBA_ERR_SHAPE;
    // padding: every token starts its own sequence (index 0), so it touches nothing
    std::fill(position_indices, position_indices + n_rows * seqlen, 0);
    for (int64_t i = 0; i < n_pieces; ++i) {
        const packmamba_piece& q = pieces[i];
        if (q.row < 0 || q.row >= n_rows || q.offset < 0 || q.length <= 0 || q.first_pos < 0 ||
            q.offset + q.length > seqlen || q.first_pos + q.length > INT32_MAX)
            return PACKMAMBA_ERR_SHAPE;
        int32_t* r = position_indices + q.row * seqlen + q.offset;
        for (int64_t t = 0; t < q.length; ++t) r[t] = (int32_t)(q.first_pos + t);
    }
    return PACKMAMBA_OK;
}

}  // extern "C"
