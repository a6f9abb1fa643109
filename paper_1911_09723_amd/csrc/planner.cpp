// Host-side format planner: validation, row ordering, bundling, wave
// balancing and packing.  See planner.hpp for the packed layout.
#include "planner.hpp"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <functional>
#include <numeric>
#include <queue>
#include <sstream>

namespace spconv {

uint16_t float_to_half_rne(float v) {
    uint32_t f;
    std::memcpy(&f, &v, 4);
    const uint32_t sign = (f >> 16) & 0x8000u;
    const uint32_t a = f & 0x7fffffffu;
    if (a >= 0x7f800000u)  // infinity or NaN
        return static_cast<uint16_t>(sign | (a > 0x7f800000u ? 0x7e00u : 0x7c00u));
    if (a >= 0x477ff000u)  // >= 65520: rounds past the largest finite half (65504)
        return static_cast<uint16_t>(sign | 0x7c00u);
    if (a >= 0x38800000u) {  // normal half range, |v| >= 2^-14
        const uint32_t m = a - 0x38000000u;  // exponent bias 127 -> 15
        uint32_t r = m >> 13;
        const uint32_t rem = m & 0x1fffu;
        if (rem > 0x1000u || (rem == 0x1000u && (r & 1u)))
            ++r;  // a mantissa carry correctly bumps the exponent
        return static_cast<uint16_t>(sign | r);
    }
    if (a < 0x33000000u)  // below 2^-25: rounds to zero (2^-25 itself ties to even zero)
        return static_cast<uint16_t>(sign);
    // subnormal half: value = mant * 2^(e - 150); in units of 2^-24 that is mant >> (126 - e)
    const uint32_t e = a >> 23;
    const uint32_t mant = (a & 0x7fffffu) | 0x800000u;
    const uint32_t shift = 126u - e;
    uint32_t r = mant >> shift;
    const uint32_t rem = mant & ((1u << shift) - 1u);
    const uint32_t half = 1u << (shift - 1u);
    if (rem > half || (rem == half && (r & 1u)))
        ++r;
    return static_cast<uint16_t>(sign | r);
}

float half_to_float(uint16_t h) {
    const int sign = (h >> 15) & 1;
    const int expo = (h >> 10) & 0x1f;
    const int frac = h & 0x3ff;
    float v;
    if (expo == 0)
        v = std::ldexp(static_cast<float>(frac), -24);
    else if (expo == 31)
        v = frac ? NAN : INFINITY;
    else
        v = std::ldexp(static_cast<float>(frac | 0x400), expo - 25);
    return sign ? -v : v;
}

Status validate(const Input &in, std::string &err) {
    std::ostringstream os;
    if (in.act < 0 || in.act > 2) {
        err = "act must be SPCONV_ACT_NONE, _RELU or _RELU6";
        return E_ARG;
    }
    if (in.storage < 0 || in.storage > 1) {
        err = "storage must be SPCONV_F32 or SPCONV_F16";
        return E_ARG;
    }
    if (in.block_rows <= 0) {
        err = "block_rows must be positive";
        return E_ARG;
    }
    if (in.block_rows != 1 && in.block_rows != 4) {
        os << "block_rows = " << in.block_rows << " is not supported (1 or 4)";
        err = os.str();
        return E_UNSUPPORTED;
    }
    if (in.cout <= 0 || in.cin <= 0) {
        os << "cout and cin must be >= 1 (got cout = " << in.cout << ", cin = " << in.cin << ")";
        err = os.str();
        return E_SHAPE;
    }
    if (in.cout % in.block_rows) {
        os << "cout = " << in.cout << " is not a multiple of block_rows = " << in.block_rows;
        err = os.str();
        return E_SHAPE;
    }
    if (in.cin > (1 << 24)) {
        err = "cin must be at most 2^24";
        return E_SHAPE;
    }
    if (!in.row_ptr) {
        err = "row_ptr is NULL";
        return E_ARG;
    }
    const int32_t rows = in.cout / in.block_rows;
    if (in.row_ptr[0] != 0) {
        os << "row_ptr[0] = " << in.row_ptr[0] << ", expected 0";
        err = os.str();
        return E_FORMAT;
    }
    for (int32_t r = 0; r < rows; ++r) {
        if (in.row_ptr[r + 1] < in.row_ptr[r]) {
            os << "row_ptr decreases at block row " << r << " (" << in.row_ptr[r] << " -> "
               << in.row_ptr[r + 1] << ")";
            err = os.str();
            return E_FORMAT;
        }
        if (in.row_ptr[r + 1] - in.row_ptr[r] > in.cin) {
            os << "block row " << r << " has " << (in.row_ptr[r + 1] - in.row_ptr[r])
               << " entries but cin = " << in.cin;
            err = os.str();
            return E_FORMAT;
        }
    }
    const int64_t nnzb = in.row_ptr[rows];
    if (nnzb > 0 && (!in.col_idx || !in.values)) {
        err = "col_idx or values is NULL but the matrix has stored entries";
        return E_ARG;
    }
    if (nnzb * static_cast<int64_t>(in.block_rows) > (int64_t(1) << 30)) {
        err = "too many stored values (limit 2^30)";
        return E_SHAPE;
    }
    for (int32_t r = 0; r < rows; ++r) {
        for (int32_t t = in.row_ptr[r]; t < in.row_ptr[r + 1]; ++t) {
            const int32_t c = in.col_idx[t];
            if (c < 0 || c >= in.cin) {
                os << "col_idx[" << t << "] = " << c << " is outside [0, " << in.cin << ") in block row " << r;
                err = os.str();
                return E_FORMAT;
            }
            if (t > in.row_ptr[r] && c <= in.col_idx[t - 1]) {
                os << "col_idx not strictly ascending in block row " << r << " at entry " << t << " ("
                   << in.col_idx[t - 1] << ", " << c << ")";
                err = os.str();
                return E_FORMAT;
            }
        }
    }
    for (int64_t i = 0; i < nnzb * in.block_rows; ++i) {
        if (!std::isfinite(in.values[i])) {
            os << "values[" << i << "] is not finite";
            err = os.str();
            return E_FORMAT;
        }
    }
    if (in.bias) {
        for (int32_t r = 0; r < in.cout; ++r) {
            if (!std::isfinite(in.bias[r])) {
                os << "bias[" << r << "] is not finite";
                err = os.str();
                return E_FORMAT;
            }
        }
    }
    return OK;
}

namespace {

// Per-bundle fixed cost (epilogue, table reads) in units of one slot step.
constexpr int64_t kBundleOverhead = 3;

// Bytes of the per-bundle table the strip kernel keeps in LDS, 16-byte rounded.
int64_t table_bytes(const Input &in) {
    const int64_t rows = in.cout / in.block_rows;
    const int64_t bundles = (rows + kGroups - 1) / kGroups;
    return (bundles * (kGroups * (1 + in.block_rows) + 1) * 4 + 15) & ~int64_t(15);
}

Status choose_geometry(const Input &in, const Options &opt, PackedPlan &p, std::string &err) {
    const int e = in.storage == 1 ? 2 : 4;
    // One strip row is 16 lanes x vec_bytes: 256 bytes read by 16 lanes at a
    // time touch all 64 LDS banks once.  Wider inputs fall back to 128-byte
    // rows, then to the direct-load kernel, which keeps 16-byte vectors.
    auto strip_bytes = [&](int vb) { return static_cast<int64_t>(in.cin) * kLanesPerRow * vb; };
    auto fits = [&](int vb) { return strip_bytes(vb) + table_bytes(in) <= kMaxLdsBytes; };
    int vb = opt.vec_bytes;
    bool strip;
    if (opt.kernel == 2) {
        strip = false;
        if (vb == 0)
            vb = 16;
    } else if (vb == 0) {
        vb = fits(16) ? 16 : 8;
        strip = fits(vb);
        if (!strip)
            vb = 16;
        if (opt.kernel == 1 && !strip) {
            err = "the X strip of cin = " + std::to_string(in.cin) + " channels does not fit in LDS";
            return E_UNSUPPORTED;
        }
    } else {
        strip = fits(vb);
        if (!strip && opt.kernel == 1) {
            err = "the X strip of cin = " + std::to_string(in.cin) + " channels at vec_bytes = " +
                  std::to_string(vb) + " does not fit in LDS";
            return E_UNSUPPORTED;
        }
    }
    p.vec_bytes = vb;
    p.cols_per_lane = vb / e;
    p.tile_cols = kLanesPerRow * p.cols_per_lane;
    if (strip) {
        p.kernel = KERNEL_STRIP;
        p.row_scale = kLanesPerRow * vb;
        p.strip_bytes = static_cast<int32_t>(strip_bytes(vb));
        p.lds_bytes = static_cast<int32_t>(strip_bytes(vb) + table_bytes(in));
        p.loader_waves = opt.prefetch ? static_cast<int32_t>((strip_bytes(vb) + kLoaderBytesPerWave - 1) /
                                                             kLoaderBytesPerWave)
                                      : 0;
    } else {
        p.kernel = KERNEL_DIRECT;
        p.row_scale = 1;
        p.strip_bytes = 0;
        p.lds_bytes = 0;
        p.loader_waves = 0;
    }
    return OK;
}

}  // namespace

Status build_plan(const Input &in, const Options &opt, PackedPlan &p, std::string &err) {
    Status st = validate(in, err);
    if (st != OK)
        return st;
    if (opt.kernel < 0 || opt.kernel > 2) {
        err = "kernel must be 0 (automatic), 1 (strip) or 2 (direct)";
        return E_ARG;
    }
    if (opt.vec_bytes != 0 && opt.vec_bytes != 8 && opt.vec_bytes != 16) {
        err = "vec_bytes must be 0, 8 or 16";
        return E_ARG;
    }
    if (opt.kernel == 2 && opt.vec_bytes == 8) {
        err = "the direct kernel reads 16-byte vectors (vec_bytes 0 or 16)";
        return E_ARG;
    }
    if (opt.waves < 0 || opt.waves > kMaxWaves) {
        err = "waves must be in [0, 16]";
        return E_ARG;
    }
    if (opt.reorder != 0 && opt.reorder != 1) {
        err = "reorder must be 0 or 1";
        return E_ARG;
    }
    if (opt.prefetch != 0 && opt.prefetch != 1) {
        err = "prefetch must be 0 or 1";
        return E_ARG;
    }

    p = PackedPlan();
    p.cout = in.cout;
    p.cin = in.cin;
    p.k = in.block_rows;
    p.act = in.act;
    p.storage = in.storage;
    st = choose_geometry(in, opt, p, err);
    if (st != OK)
        return st;

    const int32_t k = in.block_rows;
    const int32_t rows = in.cout / k;
    constexpr int32_t G = kGroups;
    p.nnzb = in.row_ptr[rows];

    // 1. processing order: descending nonzero count, ties by row index (stable)
    p.perm.resize(rows);
    std::iota(p.perm.begin(), p.perm.end(), 0);
    auto len = [&](int32_t r) { return in.row_ptr[r + 1] - in.row_ptr[r]; };
    if (opt.reorder)
        std::stable_sort(p.perm.begin(), p.perm.end(), [&](int32_t a, int32_t b) { return len(a) > len(b); });

    // 2. bundles of G consecutive rows in that order, each a whole number of
    // steps of 4 slots and at least one step long
    p.row_nnz.resize(rows);
    for (int32_t r = 0; r < rows; ++r)
        p.row_nnz[r] = len(r);
    const int32_t nb = (rows + G - 1) / G;
    std::vector<int32_t> bsteps(nb, 0);
    for (int32_t b = 0; b < nb; ++b) {
        int32_t l = 0;
        for (int32_t g = 0; g < G && b * G + g < rows; ++g)
            l = std::max(l, len(p.perm[b * G + g]));
        bsteps[b] = std::max<int32_t>(1, (l + 3) / 4);
    }

    // 3. longest-processing-time-first assignment of bundles to waves
    const int32_t max_waves = kMaxWaves - p.loader_waves;
    if (opt.waves > max_waves) {
        err = "waves = " + std::to_string(opt.waves) + " plus " + std::to_string(p.loader_waves) +
              " loader waves exceeds " + std::to_string(kMaxWaves) + " wavefronts per workgroup";
        return E_ARG;
    }
    const int32_t waves = opt.waves ? opt.waves : std::min<int32_t>(max_waves, std::max<int32_t>(nb, 1));
    p.waves = waves;
    std::vector<int32_t> order(nb);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return bsteps[a] > bsteps[b]; });
    using Item = std::pair<int64_t, int32_t>;  // (load, wave)
    std::priority_queue<Item, std::vector<Item>, std::greater<Item>> heap;
    for (int32_t w = 0; w < waves; ++w)
        heap.push({0, w});
    std::vector<std::vector<int32_t>> lists(waves);
    std::vector<int64_t> load(waves, 0);
    for (int32_t b : order) {
        Item it = heap.top();
        heap.pop();
        lists[it.second].push_back(b);
        it.first += 4 * static_cast<int64_t>(bsteps[b]) + kBundleOverhead;
        load[it.second] = it.first;
        heap.push(it);
    }
    p.max_wave_cost = waves ? *std::max_element(load.begin(), load.end()) : 0;
    p.sum_wave_cost = std::accumulate(load.begin(), load.end(), int64_t(0));

    // 4. pack: bundles in wave order; each wave's steps in chunks of 4 steps
    p.wave_ptr.assign(waves + 1, 0);
    p.wave_chunk.assign(waves + 1, 0);
    p.split.assign(static_cast<size_t>(waves) * (kMaxParts + 1), 0);
    p.hdr.reserve(2 * static_cast<size_t>(nb));
    p.rows.reserve(static_cast<size_t>(G) * nb);
    p.bundle_bias.reserve(static_cast<size_t>(G) * nb * k);
    int64_t chunk0 = 0;  // first chunk of the current wave
    int32_t bglob = 0;   // bundles packed so far
    int32_t max_bundles = 0;
    for (int32_t w = 0; w < waves; ++w) {
        int64_t total = 0;
        for (int32_t b : lists[w])
            total += bsteps[b];
        const int64_t nchunks = (total + kChunkSteps - 1) / kChunkSteps;
        if ((chunk0 + nchunks) * 64 * k > (int64_t(1) << 29)) {  // stream byte sizes stay below 2^31
            err = "packed plan too large";
            return E_SHAPE;
        }
        p.idx.resize(static_cast<size_t>((chunk0 + nchunks) * 64), 0);
        p.val.resize(static_cast<size_t>((chunk0 + nchunks) * 64 * k), 0.0f);
        // split[i]: first bundle whose first step is at or after i/64 of the stream
        std::vector<int64_t> start(lists[w].size() + 1, 0);
        for (size_t i = 0; i < lists[w].size(); ++i)
            start[i + 1] = start[i] + bsteps[lists[w][i]];
        for (int32_t i = 0; i <= kMaxParts; ++i) {
            size_t j = 0;
            while (j < lists[w].size() && start[j] * kMaxParts < static_cast<int64_t>(i) * total)
                ++j;
            if (i == kMaxParts)
                j = lists[w].size();
            p.split[static_cast<size_t>(w) * (kMaxParts + 1) + i] = bglob + static_cast<int32_t>(j);
        }
        for (size_t i = 0; i < lists[w].size(); ++i) {
            const int32_t b = lists[w][i];
            const int64_t s_first = start[i];
            p.hdr.push_back(static_cast<int32_t>(s_first));
            p.hdr.push_back(bsteps[b]);
            for (int32_t g = 0; g < G; ++g) {
                const int32_t pos = b * G + g;
                const int32_t rb = pos < rows ? p.perm[pos] : -1;
                p.rows.push_back(rb);
                for (int32_t ii = 0; ii < k; ++ii)
                    p.bundle_bias.push_back(rb >= 0 && in.bias ? in.bias[rb * k + ii] : 0.0f);
                if (rb < 0)
                    continue;
                const int32_t r0 = in.row_ptr[rb];
                for (int32_t t = 0; t < len(rb); ++t) {
                    const int64_t s = s_first + t / 4;
                    const int64_t e = 64 * (chunk0 + s / kChunkSteps) + kLanesPerRow * g + 4 * (s % kChunkSteps) +
                                      (t % 4);
                    p.idx[e] = in.col_idx[r0 + t] * p.row_scale;
                    for (int32_t ii = 0; ii < k; ++ii) {
                        float v = in.values[static_cast<int64_t>(r0 + t) * k + ii];
                        if (in.storage == 1)
                            v = half_to_float(float_to_half_rne(v));
                        p.val[e * k + ii] = v;
                    }
                }
            }
        }
        bglob += static_cast<int32_t>(lists[w].size());
        max_bundles = std::max<int32_t>(max_bundles, static_cast<int32_t>(lists[w].size()));
        p.wave_ptr[w + 1] = bglob;
        chunk0 += nchunks;
        p.wave_chunk[w + 1] = static_cast<int32_t>(chunk0);
    }
    p.slots = chunk0 * 64;
    // A tile is shared by at most as many workgroups as the busiest wave has bundles.
    p.max_parts = 1;
    while (p.max_parts * 2 <= std::min<int32_t>(kMaxParts, max_bundles))
        p.max_parts *= 2;
    return OK;
}

void unpack_plan(const PackedPlan &p, int32_t *row_ptr, int32_t *col_idx, float *values, int32_t *perm) {
    const int32_t k = p.k;
    const int32_t rows = p.cout / k;
    constexpr int32_t G = kGroups;
    std::vector<std::vector<int32_t>> cols(rows);
    std::vector<std::vector<float>> vals(rows);
    const int32_t waves = static_cast<int32_t>(p.wave_ptr.size()) - 1;
    // each row's real entries are the first row_nnz[rb] slots of its sequence
    for (int32_t w = 0; w < waves; ++w) {
        for (int32_t b = p.wave_ptr[w]; b < p.wave_ptr[w + 1]; ++b) {
            const int64_t s_first = p.hdr[2 * b];
            for (int32_t g = 0; g < G; ++g) {
                const int32_t rb = p.rows[static_cast<size_t>(b) * G + g];
                if (rb < 0)
                    continue;
                for (int32_t t = 0; t < p.row_nnz[rb]; ++t) {
                    const int64_t s = s_first + t / 4;
                    const int64_t e = 64 * (p.wave_chunk[w] + s / kChunkSteps) + kLanesPerRow * g +
                                      4 * (s % kChunkSteps) + (t % 4);
                    cols[rb].push_back(p.idx[e] / p.row_scale);
                    for (int32_t i = 0; i < k; ++i)
                        vals[rb].push_back(p.val[e * k + i]);
                }
            }
        }
    }
    int32_t acc = 0;
    if (row_ptr)
        row_ptr[0] = 0;
    for (int32_t r = 0; r < rows; ++r) {
        if (col_idx)
            std::copy(cols[r].begin(), cols[r].end(), col_idx + acc);
        if (values)
            std::copy(vals[r].begin(), vals[r].end(), values + static_cast<int64_t>(acc) * k);
        acc += static_cast<int32_t>(cols[r].size());
        if (row_ptr)
            row_ptr[r + 1] = acc;
    }
    if (perm)
        std::copy(p.perm.begin(), p.perm.end(), perm);
}

}  // namespace spconv
