// planner.cpp -- host planning of a cross-mesh resharding task (no HIP calls).
#include "planner.hpp"

#include <algorithm>
#include <map>
#include <numeric>

namespace rs {

// ---------------------------------------------------------------- parsing
// Section 2.2, "Sharding spec": one letter per tensor dim, R or S with the
// mesh dims the tensor dim is split along.  Accepts S^0, S_0, S^{01}, S01.
std::string parse_spec(const char *spec, int ndim, int mesh_ndim, std::vector<std::vector<int>> &axes) {
    axes.clear();
    if (!spec) return "spec is NULL";
    const std::string s(spec);
    size_t i = 0;
    auto skip = [&]() { while (i < s.size() && (s[i] == ' ' || s[i] == ',' || s[i] == '\t')) ++i; };
    skip();
    while (i < s.size()) {
        const char c = s[i];
        if (c == 'R') {
            axes.emplace_back();
            ++i;
        } else if (c == 'S') {
            ++i;
            if (i < s.size() && (s[i] == '^' || s[i] == '_')) ++i;
            bool brace = false;
            if (i < s.size() && s[i] == '{') { brace = true; ++i; }
            std::vector<int> a;
            while (i < s.size() && s[i] >= '0' && s[i] <= '9') a.push_back(s[i++] - '0');
            if (a.empty()) return "spec '" + s + "': S without mesh axes";
            if (brace) {
                if (i >= s.size() || s[i] != '}') return "spec '" + s + "': missing '}'";
                ++i;
            }
            axes.push_back(std::move(a));
        } else {
            return "spec '" + s + "': unexpected character '" + std::string(1, c) + "'";
        }
        skip();
    }
    if (int(axes.size()) != ndim)
        return "spec '" + s + "' has " + std::to_string(axes.size()) + " letters but the tensor has " +
               std::to_string(ndim) + " dims";
    std::vector<int> used(10, 0);
    for (auto &a : axes)
        for (int x : a) {
            if (x >= mesh_ndim)
                return "spec '" + s + "' names mesh axis " + std::to_string(x) + " but the mesh has " +
                       std::to_string(mesh_ndim) + " axes";
            if (used[x]++) return "spec '" + s + "' uses mesh axis " + std::to_string(x) + " twice";
        }
    return "";
}

// ----------------------------------------------------------------- layout
std::string build_layout(const std::vector<int64_t> &shape, const std::vector<int64_t> &mesh,
                         const std::vector<std::vector<int>> &axes, Layout &L) {
    const int nd = int(shape.size());
    L.mesh = mesh;
    L.axes = axes;
    L.ndev = 1;
    for (int64_t m : mesh) L.ndev *= m;
    L.nshards.assign(nd, 1);
    L.bounds.assign(nd, {});
    for (int d = 0; d < nd; ++d) {
        int64_t k = 1;
        for (int a : axes[d]) k *= mesh[a];
        L.nshards[d] = k;
        // balanced split: the first (l mod k) shards are one element longer
        const int64_t l = shape[d], q = l / k, r = l % k;
        auto &b = L.bounds[d];
        b.resize(k + 1);
        for (int64_t j = 0; j <= k; ++j) b[j] = j * q + std::min(j, r);
    }
    // device -> shard index per dim (row-major device numbering; axis list major to minor)
    const int md = int(mesh.size());
    L.dev_shard.assign(L.ndev * nd, 0);
    std::vector<int64_t> c(md);
    for (int64_t dev = 0; dev < L.ndev; ++dev) {
        int64_t rem = dev;
        for (int a = md - 1; a >= 0; --a) { c[a] = rem % mesh[a]; rem /= mesh[a]; }
        for (int d = 0; d < nd; ++d) {
            int64_t j = 0;
            for (int a : axes[d]) j = j * mesh[a] + c[a];
            L.dev_shard[dev * nd + d] = j;
        }
    }
    // CSR: linearised shard tuple -> holders
    int64_t nlin = 1;
    for (int d = 0; d < nd; ++d) nlin *= L.nshards[d];
    std::vector<int64_t> lin(L.ndev);
    L.shard_devs_off.assign(nlin + 1, 0);
    for (int64_t dev = 0; dev < L.ndev; ++dev) {
        int64_t x = 0;
        for (int d = 0; d < nd; ++d) x = x * L.nshards[d] + L.dev_shard[dev * nd + d];
        lin[dev] = x;
        L.shard_devs_off[x + 1]++;
    }
    for (int64_t x = 0; x < nlin; ++x) L.shard_devs_off[x + 1] += L.shard_devs_off[x];
    L.shard_devs.assign(L.ndev, 0);
    std::vector<int64_t> fill(L.shard_devs_off.begin(), L.shard_devs_off.end() - 1);
    for (int64_t dev = 0; dev < L.ndev; ++dev) L.shard_devs[fill[lin[dev]]++] = int32_t(dev);
    return "";
}

// ------------------------------------------------------------- unit tasks
namespace {
struct Overlap {
    int64_t lo, hi, js, jd;
};
}  // namespace

void build_tasks(Plan &p) {
    const int nd = p.ndim;
    std::vector<std::vector<Overlap>> per(nd);
    for (int d = 0; d < nd; ++d) {
        const auto &bs = p.src.bounds[d], &bd = p.dst.bounds[d];
        const int64_t ks = p.src.nshards[d], kd = p.dst.nshards[d];
        int64_t i = 0, j = 0;
        while (i < ks && j < kd) {
            const int64_t lo = std::max(bs[i], bd[j]), hi = std::min(bs[i + 1], bd[j + 1]);
            if (lo < hi) per[d].push_back({lo, hi, i, j});
            if (bs[i + 1] <= bd[j + 1]) ++i; else ++j;
        }
    }
    p.tasks.clear();
    for (int d = 0; d < nd; ++d)
        if (per[d].empty()) return;
    std::vector<size_t> idx(nd, 0);
    for (;;) {
        UnitTask t;
        t.lo.resize(nd);
        t.hi.resize(nd);
        int64_t vol = 1, xs = 0, xd = 0;
        for (int d = 0; d < nd; ++d) {
            const Overlap &o = per[d][idx[d]];
            t.lo[d] = o.lo;
            t.hi[d] = o.hi;
            vol *= o.hi - o.lo;
            xs = xs * p.src.nshards[d] + o.js;
            xd = xd * p.dst.nshards[d] + o.jd;
        }
        t.src_shard = xs;
        t.dst_shard = xd;
        t.bytes = vol * p.es;
        p.tasks.push_back(std::move(t));
        int d = nd - 1;
        while (d >= 0 && ++idx[d] == per[d].size()) idx[d--] = 0;
        if (d < 0) break;
    }
}

// ----------------------------------------------------------- sender choice
void choose_senders(Plan &p) {
    const auto &off = p.src.shard_devs_off;
    const auto &devs = p.src.shard_devs;
    if (p.flags & 0x1u) {  // naive: lowest-indexed owner
        for (auto &t : p.tasks) t.sender = devs[off[t.src_shard]];
        return;
    }
    // Eq. 4: tasks longest first (ties keep task order), each to the owner
    // with the least bytes assigned so far (ties: lowest device index).
    std::vector<size_t> order(p.tasks.size());
    std::iota(order.begin(), order.end(), size_t(0));
    std::stable_sort(order.begin(), order.end(),
                     [&](size_t a, size_t b) { return p.tasks[a].bytes > p.tasks[b].bytes; });
    std::vector<int64_t> load(p.src.ndev, 0);
    for (size_t i : order) {
        auto &t = p.tasks[i];
        int32_t best = -1;
        for (int64_t k = off[t.src_shard]; k < off[t.src_shard + 1]; ++k) {
            const int32_t dev = devs[k];  // ascending, so strict < keeps the lowest index on ties
            if (best < 0 || load[dev] < load[best]) best = dev;
        }
        t.sender = best;
        load[best] += t.bytes;
    }
}

// ---------------------------------------------------------------- lowering
namespace {

struct Level {
    int64_t n, ss, ds;  // extent, sender byte stride, receiver byte stride
};

struct Piece {
    uint64_t src_off, dst_off;
    int64_t run;               // bytes, contiguous on both sides
    std::vector<Level> outer;  // outermost first, at most 3
    int32_t w;                 // vector bytes
    bool realign = false;      // rows in different 16-byte phases: LDS path
};

// Rows of at least this many bytes whose source and destination 16-byte
// phases differ take the LDS realignment path; they are cut into segments of
// at most kRealignSeg bytes so a pass over a few rows fits the staging area.
constexpr int64_t kRealignMinRun = 64;
constexpr int64_t kRealignSeg = 4096;

int64_t pow2_divisor(int64_t x, int64_t cap) {
    int64_t w = cap;
    while (w > 1 && (x % w) != 0) w >>= 1;
    return w;
}

int32_t pick_width(uint64_t so, uint64_t dso, int64_t run, const std::vector<Level> &outer) {
    int64_t w = 16;
    w = pow2_divisor(int64_t(so), w);
    w = pow2_divisor(int64_t(dso), w);
    w = pow2_divisor(run, w);
    for (const auto &l : outer) {
        w = pow2_divisor(l.ss, w);
        w = pow2_divisor(l.ds, w);
    }
    return int32_t(w);
}

constexpr uint64_t kMaxPieceVectors = (uint64_t(1) << 31) - 1;
constexpr uint64_t kMaxDescs = uint64_t(1) << 24;  // 1.75 GiB of descriptors

// Index units per row: vectors on the direct path, whole rows on the
// realignment path.
uint64_t units_per_row(const Piece &pc) { return pc.realign ? 1 : uint64_t(pc.run / pc.w); }

// 64-bit byte offsets (sender, receiver) of vector v of a piece.
std::pair<uint64_t, uint64_t> piece_off64(const Piece &pc, uint64_t vpr, uint64_t v) {
    uint64_t row = v / vpr;
    const uint64_t col = v - row * vpr;
    uint64_t s = pc.src_off + col * uint64_t(pc.w), t = pc.dst_off + col * uint64_t(pc.w);
    const int nl = int(pc.outer.size());
    for (int i = nl - 1; i >= 0; --i) {
        const uint64_t n = uint64_t(pc.outer[i].n);
        const uint64_t idx = i == 0 ? row : row % n;
        s += idx * uint64_t(pc.outer[i].ss);
        t += idx * uint64_t(pc.outer[i].ds);
        row = i == 0 ? 0 : row / n;
    }
    return {s, t};
}

constexpr uint64_t kMaxChunkSpan = uint64_t(1) << 32;

// Byte extents (end of the last byte from the origin) of a piece on the two
// sides.
std::pair<uint64_t, uint64_t> piece_span(const Piece &pc) {
    uint64_t es_ = uint64_t(pc.run), ed = uint64_t(pc.run);
    for (const auto &l : pc.outer) {
        es_ += uint64_t(l.n - 1) * uint64_t(l.ss);
        ed += uint64_t(l.n - 1) * uint64_t(l.ds);
    }
    return {es_, ed};
}

// Whether offsets grow with the vector index on both sides: every level's
// stride is at least the extent of everything inside it.  Plain (unpermuted)
// layouts always are; a permuted one need not be, and its chunks then take
// the piece's origin as their base (every offset of a piece is at or above
// its origin, strides being non-negative).
bool monotone(const Piece &pc) {
    uint64_t es_ = uint64_t(pc.run), ed = uint64_t(pc.run);
    for (size_t i = pc.outer.size(); i-- > 0;) {
        const Level &l = pc.outer[i];
        if (uint64_t(l.ss) < es_ || uint64_t(l.ds) < ed) return false;
        es_ += uint64_t(l.n - 1) * uint64_t(l.ss);
        ed += uint64_t(l.n - 1) * uint64_t(l.ds);
    }
    return true;
}

// Whether the chunks of a piece (from 0 to n, each ending where next_end
// says) fit in the descriptor budget.  Counts without building any, so a
// piece cut into too many chunks fails before it takes memory.
template <class F>
bool fits_chunk_budget(Plan &p, uint64_t n, F next_end) {
    uint64_t k = p.descs.size();
    for (uint64_t x = 0; x < n; x = next_end(x))
        if (++k > kMaxDescs) {
            p.too_many = true;
            return false;
        }
    return true;
}

// Realignment path: chunks are ranges of whole rows.
void emit_realign(Plan &p, const Piece &pc, int32_t src_buf, int64_t fan_off, int64_t nfan, int64_t chunk_bytes) {
    Desc d{};
    const int nl = int(pc.outer.size());
    const int levels = std::max(1, nl);
    for (int i = 0; i < nl; ++i) {
        const Level &l = pc.outer[nl - 1 - i];
        d.ss[i] = uint32_t(uint64_t(l.ss));
        d.ds[i] = uint32_t(uint64_t(l.ds));
    }
    uint64_t rows = 1;
    for (const auto &l : pc.outer) rows *= uint64_t(l.n);
    const uint32_t m = realign_words(uint32_t(pc.run));
    d.run = uint32_t(pc.run);
    d.vpr = m;
    d.batch = std::max<uint32_t>(1, kRealignStageBytes / (m * 16u));
    d.n1 = nl >= 2 ? uint32_t(pc.outer[nl - 1].n) : 1u;
    d.n2 = nl >= 3 ? uint32_t(pc.outer[nl - 2].n) : 1u;
    const FastDiv f0 = make_fastdiv(m), f1 = make_fastdiv(d.n1), f2 = make_fastdiv(d.n2);
    d.mul_vpr = f0.mul; d.sh_vpr = uint8_t(f0.shift);
    d.mul_n1 = f1.mul;  d.sh_n1 = uint8_t(f1.shift);
    d.mul_n2 = f2.mul;  d.sh_n2 = uint8_t(f2.shift);
    d.kind = uint8_t(make_kind(4, uint32_t(levels)) | kRealign);
    d.src_buf = uint16_t(src_buf);
    d.nfan = uint16_t(nfan);
    d.fan_off = uint32_t(fan_off);
    const uint64_t cr = uint64_t(std::max<int64_t>(1, chunk_bytes / pc.run));  // rows per chunk
    if (p.descs.size() + (rows + cr - 1) / cr > kMaxDescs) {
        p.too_many = true;
        return;
    }
    const bool mono = monotone(pc);
    // end of the chunk from row r0: cr rows, fewer where they would span
    // 2^31 bytes (the kernel forms signed 32-bit word offsets)
    auto chunk_end = [&](uint64_t r0, const std::pair<uint64_t, uint64_t> &first) {
        uint64_t r1 = std::min(rows, r0 + cr);
        for (; mono;) {
            const auto last = piece_off64(pc, 1, r1 - 1);
            if (last.first + uint64_t(pc.run) - first.first < kMaxChunkSpan / 2 &&
                last.second + uint64_t(pc.run) - first.second < kMaxChunkSpan / 2)
                break;
            r1 = r0 + (r1 - r0) / 2;
        }
        return r1;
    };
    if (mono && p.descs.size() + rows > kMaxDescs && !fits_chunk_budget(p, rows, [&](uint64_t r0) {
            return chunk_end(r0, piece_off64(pc, 1, r0));
        }))
        return;
    for (uint64_t r0 = 0; r0 < rows;) {
        const auto first = mono ? piece_off64(pc, 1, r0) : std::pair<uint64_t, uint64_t>(pc.src_off, pc.dst_off);
        const uint64_t r1 = chunk_end(r0, first);
        if (p.descs.size() >= kMaxDescs) {
            p.too_many = true;
            return;
        }
        d.v0 = uint32_t(r0);
        d.v1 = uint32_t(r1);
        d.src_base = first.first;
        d.dst_base = first.second;
        d.src_rel0 = uint32_t(first.first - pc.src_off);
        d.dst_rel0 = uint32_t(first.second - pc.dst_off);
        p.descs.push_back(d);
        r0 = r1;
    }
    p.align = std::max<int64_t>(p.align, 16);
    p.lds_bytes = std::max(p.lds_bytes, realign_lds_bytes(d.batch, m));
}

// Emit chunks of a piece whose outer list has at most 3 levels and fewer
// than 2^31 vectors.  Every chunk spans less than 2^32 bytes on both sides.
void emit(Plan &p, const Piece &pc, int32_t src_buf, int64_t fan_off, int64_t nfan, int64_t chunk_bytes) {
    if (pc.realign) {
        emit_realign(p, pc, src_buf, fan_off, nfan, chunk_bytes);
        return;
    }
    Desc d{};
    const int nl = int(pc.outer.size());
    const int levels = std::max(1, nl);
    // outer[] is outermost first; Desc level 1 is the innermost outer level
    for (int i = 0; i < nl; ++i) {
        const Level &l = pc.outer[nl - 1 - i];
        d.ss[i] = uint32_t(uint64_t(l.ss));
        d.ds[i] = uint32_t(uint64_t(l.ds));
    }
    const uint64_t vpr = uint64_t(pc.run / pc.w);
    uint64_t rows = 1;
    for (const auto &l : pc.outer) rows *= uint64_t(l.n);
    const uint64_t total = vpr * rows;
    d.vpr = uint32_t(vpr);
    d.n1 = nl >= 2 ? uint32_t(pc.outer[nl - 1].n) : 1u;
    d.n2 = nl >= 3 ? uint32_t(pc.outer[nl - 2].n) : 1u;
    const FastDiv f0 = make_fastdiv(d.vpr), f1 = make_fastdiv(d.n1), f2 = make_fastdiv(d.n2);
    d.mul_vpr = f0.mul; d.sh_vpr = uint8_t(f0.shift);
    d.mul_n1 = f1.mul;  d.sh_n1 = uint8_t(f1.shift);
    d.mul_n2 = f2.mul;  d.sh_n2 = uint8_t(f2.shift);
    uint32_t log2w = 0;
    while ((1 << log2w) < pc.w) ++log2w;
    d.kind = uint8_t(make_kind(log2w, uint32_t(levels)));
    d.src_buf = uint16_t(src_buf);
    d.nfan = uint16_t(nfan);
    d.fan_off = uint32_t(fan_off);
    // chunk length in vectors: whole 256-byte groups where the width allows
    uint64_t cv = uint64_t(std::max<int64_t>(1, chunk_bytes / pc.w));
    const uint64_t grain = uint64_t(256 / pc.w);
    cv = std::max(grain, cv / grain * grain);
    if (p.descs.size() + (total + cv - 1) / cv > kMaxDescs) {
        p.too_many = true;
        return;
    }
    const bool mono = monotone(pc);
    // end of the chunk from vector v0: cv vectors, fewer where they would
    // span 2^32 bytes on either side
    auto chunk_end = [&](uint64_t v0, const std::pair<uint64_t, uint64_t> &first) {
        uint64_t v1 = std::min(total, v0 + cv);
        for (; mono;) {
            const auto last = piece_off64(pc, vpr, v1 - 1);
            if (last.first + uint64_t(pc.w) - first.first < kMaxChunkSpan &&
                last.second + uint64_t(pc.w) - first.second < kMaxChunkSpan)
                break;
            v1 = v0 + (v1 - v0) / 2;
        }
        return v1;
    };
    if (mono && p.descs.size() + total > kMaxDescs && !fits_chunk_budget(p, total, [&](uint64_t v0) {
            return chunk_end(v0, piece_off64(pc, vpr, v0));
        }))
        return;
    for (uint64_t v0 = 0; v0 < total;) {
        const auto first = mono ? piece_off64(pc, vpr, v0) : std::pair<uint64_t, uint64_t>(pc.src_off, pc.dst_off);
        const uint64_t v1 = chunk_end(v0, first);
        if (p.descs.size() >= kMaxDescs) {
            p.too_many = true;
            return;
        }
        d.v0 = uint32_t(v0);
        d.v1 = uint32_t(v1);
        d.src_base = first.first;
        d.dst_base = first.second;
        d.src_rel0 = uint32_t(first.first - pc.src_off);
        d.dst_rel0 = uint32_t(first.second - pc.dst_off);
        p.descs.push_back(d);
        v0 = v1;
    }
    p.align = std::max<int64_t>(p.align, pc.w);
}

// Emit every row of the outermost level as its own piece (level removed).
void split_emit(Plan &p, Piece pc, int32_t src_buf, int64_t fan_off, int64_t nfan, int64_t chunk_bytes);

void peel_top(Plan &p, const Piece &pc, int32_t src_buf, int64_t fan_off, int64_t nfan, int64_t chunk_bytes) {
    const Level top = pc.outer.front();
    Piece sub = pc;
    sub.outer.erase(sub.outer.begin());
    for (int64_t i = 0; i < top.n; ++i) {
        sub.src_off = pc.src_off + uint64_t(i * top.ss);
        sub.dst_off = pc.dst_off + uint64_t(i * top.ds);
        split_emit(p, sub, src_buf, fan_off, nfan, chunk_bytes);
        if (p.too_many) return;
    }
}

// Split a piece until it has at most 3 outer levels and fewer than 2^31
// vectors, then emit it.
void split_emit(Plan &p, Piece pc, int32_t src_buf, int64_t fan_off, int64_t nfan, int64_t chunk_bytes) {
    if (p.too_many) return;
    if (pc.outer.size() > 3) {
        peel_top(p, pc, src_buf, fan_off, nfan, chunk_bytes);
        return;
    }
    if (!monotone(pc)) {
        // chunks based at the piece's origin: the whole piece within 32-bit
        // offsets (31 on the realignment path, whose word offsets are signed)
        const auto sp = piece_span(pc);
        const uint64_t lim = pc.realign ? kMaxChunkSpan / 2 : kMaxChunkSpan;
        if (sp.first >= lim || sp.second >= lim) {  // (a single level is always monotone)
            peel_top(p, pc, src_buf, fan_off, nfan, chunk_bytes);
            return;
        }
    }
    uint64_t rows = 1;
    for (const auto &l : pc.outer) rows *= uint64_t(l.n);
    const uint64_t vpr = units_per_row(pc);
    const uint64_t total = vpr * rows;
    if (total <= kMaxPieceVectors) {
        emit(p, pc, src_buf, fan_off, nfan, chunk_bytes);
        return;
    }
    if (pc.outer.empty()) {
        // a single run longer than the index range: cut it into segments
        const int64_t segb = (int64_t(1) << 30) * pc.w;
        for (int64_t b = 0; b < pc.run; b += segb) {
            Piece sub = pc;
            sub.run = std::min(segb, pc.run - b);
            sub.src_off = pc.src_off + uint64_t(b);
            sub.dst_off = pc.dst_off + uint64_t(b);
            emit(p, sub, src_buf, fan_off, nfan, chunk_bytes);
        }
        return;
    }
    const Level top = pc.outer.front();
    const uint64_t inner = total / uint64_t(top.n);
    if (inner > kMaxPieceVectors) {
        peel_top(p, pc, src_buf, fan_off, nfan, chunk_bytes);
        return;
    }
    // cut the outermost level into ranges that fit
    const int64_t step = int64_t(kMaxPieceVectors / inner);
    for (int64_t i = 0; i < top.n; i += step) {
        Piece sub = pc;
        sub.outer.front().n = std::min(step, top.n - i);
        sub.src_off = pc.src_off + uint64_t(i * top.ss);
        sub.dst_off = pc.dst_off + uint64_t(i * top.ds);
        emit(p, sub, src_buf, fan_off, nfan, chunk_bytes);
    }
}

#ifndef RS_TMAXW_LOG2
#define RS_TMAXW_LOG2 2u  // widest tile along B: 4 x 128 bytes
#endif

// Tile-transpose piece (see desc.h): A contiguous in the sender's buffer, B
// in the receivers'; outer levels outermost first (any number: more than two
// are peeled into separate pieces).
struct TPiece {
    uint64_t src_off, dst_off;
    int64_t na, nb;            // extents of A and B (elements)
    int64_t ss_b, ds_a;        // sender stride of B, receiver stride of A (bytes)
    std::vector<Level> outer;  // outermost first
};

void emit_transpose(Plan &p, const TPiece &tp, int32_t src_buf, int64_t fan_off, int64_t nfan, int64_t chunk_bytes,
                    std::vector<Desc> &out) {
    if (p.too_many || p.tile_span_too_long) return;
    if (tp.outer.size() > 2) {
        const Level top = tp.outer.front();
        TPiece sub = tp;
        sub.outer.erase(sub.outer.begin());
        for (int64_t i = 0; i < top.n; ++i) {
            sub.src_off = tp.src_off + uint64_t(i * top.ss);
            sub.dst_off = tp.dst_off + uint64_t(i * top.ds);
            emit_transpose(p, sub, src_buf, fan_off, nfan, chunk_bytes, out);
            if (p.too_many || p.tile_span_too_long) return;
        }
        return;
    }
    const int64_t es = p.es;
    const int64_t te = int64_t(tile_elems(uint32_t(es)));
    {
        // every tile is addressed from the piece's origin: the piece must lie
        // within 32-bit offsets on both sides (else peel an outer level, or
        // halve A or B in whole tiles)
        uint64_t ss_ = uint64_t(tp.nb - 1) * uint64_t(tp.ss_b) + uint64_t(tp.na * es);
        uint64_t sd_ = uint64_t(tp.na - 1) * uint64_t(tp.ds_a) + uint64_t(tp.nb * es);
        for (const auto &l : tp.outer) {
            ss_ += uint64_t(l.n - 1) * uint64_t(l.ss);
            sd_ += uint64_t(l.n - 1) * uint64_t(l.ds);
        }
        if (ss_ >= kMaxChunkSpan || sd_ >= kMaxChunkSpan) {
            if (!tp.outer.empty()) {
                const Level top = tp.outer.front();
                TPiece sub = tp;
                sub.outer.erase(sub.outer.begin());
                for (int64_t i = 0; i < top.n; ++i) {
                    sub.src_off = tp.src_off + uint64_t(i * top.ss);
                    sub.dst_off = tp.dst_off + uint64_t(i * top.ds);
                    emit_transpose(p, sub, src_buf, fan_off, nfan, chunk_bytes, out);
                    if (p.too_many || p.tile_span_too_long) return;
                }
                return;
            }
            // A and B only: the source span grows with B (stride ss_b) and
            // with A's run, the destination span with A (stride ds_a) and
            // with B's run.  Halve the extent behind the larger term of the
            // span that is too long, in whole tiles (whole 4-tile groups
            // along B while it is long).
            const uint64_t sb_term = uint64_t(tp.nb - 1) * uint64_t(tp.ss_b), sa_term = uint64_t(tp.na * es);
            const uint64_t da_term = uint64_t(tp.na - 1) * uint64_t(tp.ds_a), db_term = uint64_t(tp.nb * es);
            const bool cut_b = ss_ >= kMaxChunkSpan ? sb_term >= sa_term : db_term > da_term;
            const int64_t n = cut_b ? tp.nb : tp.na;
            // One tile along that extent already too long: the caller admits
            // only pieces whose tile strides fit 31 bits, so this cannot
            // happen there; it fails the plan rather than recursing forever.
            if (n <= te) {
                p.tile_span_too_long = true;
                return;
            }
            const int64_t step = n / 2 >= 4 * te && cut_b ? 4 * te : te;
            const int64_t half = std::max<int64_t>(step, (n / 2) / step * step);
            for (int64_t x0 = 0; x0 < n; x0 += half) {
                TPiece sub = tp;
                if (cut_b) {
                    sub.nb = std::min(half, tp.nb - x0);
                    sub.src_off = tp.src_off + uint64_t(x0 * tp.ss_b);
                    sub.dst_off = tp.dst_off + uint64_t(x0 * es);
                } else {
                    sub.na = std::min(half, tp.na - x0);
                    sub.src_off = tp.src_off + uint64_t(x0 * es);
                    sub.dst_off = tp.dst_off + uint64_t(x0 * tp.ds_a);
                }
                emit_transpose(p, sub, src_buf, fan_off, nfan, chunk_bytes, out);
                if (p.too_many || p.tile_span_too_long) return;
            }
            return;
        }
    }
    const int nl = int(tp.outer.size());
    const Level o1 = nl >= 1 ? tp.outer[size_t(nl - 1)] : Level{1, 0, 0};
    const Level o2 = nl >= 2 ? tp.outer[0] : Level{1, 0, 0};
    // tile width along B: the narrowest of 1, 2, 4 x 128 bytes that covers
    // the whole B extent (a tile then writes whole destination rows), with at
    // most 256 tile rows (32 KiB of LDS); B extents wider than that take
    // 2 x 128 bytes, which keeps twice the tiles resident (measured: 512-byte
    // rows 382.6 us at 512-byte tiles against 391.6 at 256; 1 KiB rows 24.4
    // against 26.2 us the other way).  With one receiver, 2 x 128 bytes at
    // most (measured: workload 5's tensor to one replica, 512-byte rows,
    // 150.5 us against 152.6 at 512-byte tiles; with 4 replicas 512-byte
    // tiles stay ahead, 381.2 against 388.3).
    uint32_t wide = 0;
    while (wide < RS_TMAXW_LOG2 && (te << wide) < tp.nb && (te << (wide + 1)) <= 256) ++wide;
    if (((te << wide) < tp.nb || nfan == 1) && wide > 1) wide = 1;
    const int64_t tr = te << wide;
    const uint64_t ntb = uint64_t((tp.nb + tr - 1) / tr), nta = uint64_t((tp.na + te - 1) / te);
    const uint64_t tiles = ntb * nta * uint64_t(o1.n) * uint64_t(o2.n);
    Desc d{};
    bool ald = tp.src_off % 16 == 0 && tp.ss_b % 16 == 0 && o1.ss % 16 == 0 && o2.ss % 16 == 0;
    bool ast = tp.dst_off % 16 == 0 && tp.ds_a % 16 == 0 && o1.ds % 16 == 0 && o2.ds % 16 == 0;
    uint32_t log2es = 0;
    while ((int64_t(1) << log2es) < es) ++log2es;
    d.kind = uint8_t(log2es | (ald ? kTAlignLoad : 0u) | (ast ? kTAlignStore : 0u) | (wide << 6));
    d.ss[0] = uint32_t(uint64_t(tp.ss_b));
    d.ds[0] = uint32_t(uint64_t(tp.ds_a));
    d.ss[1] = uint32_t(uint64_t(o1.ss));
    d.ds[1] = uint32_t(uint64_t(o1.ds));
    d.ss[2] = uint32_t(uint64_t(o2.ss));
    d.ds[2] = uint32_t(uint64_t(o2.ds));
    d.vpr = uint32_t(ntb);
    d.n1 = uint32_t(nta);
    d.n2 = uint32_t(o1.n);
    const FastDiv f0 = make_fastdiv(d.vpr), f1 = make_fastdiv(d.n1), f2 = make_fastdiv(d.n2);
    d.mul_vpr = f0.mul; d.sh_vpr = uint8_t(f0.shift);
    d.mul_n1 = f1.mul;  d.sh_n1 = uint8_t(f1.shift);
    d.mul_n2 = f2.mul;  d.sh_n2 = uint8_t(f2.shift);
    d.run = uint32_t(tp.na);
    d.batch = uint32_t(tp.nb);
    d.src_buf = uint16_t(src_buf);
    d.nfan = uint16_t(nfan);
    d.fan_off = uint32_t(fan_off);
    const uint64_t per = uint64_t(std::max<int64_t>(1, chunk_bytes / (te * tr * es)));
    if (p.descs.size() + out.size() + (tiles + per - 1) / per > kMaxDescs) {
        p.too_many = true;
        return;
    }
    d.src_base = tp.src_off;
    d.dst_base = tp.dst_off;
    d.src_rel0 = 0;
    d.dst_rel0 = 0;
    for (uint64_t t0 = 0; t0 < tiles;) {
        const uint64_t t1 = std::min(tiles, t0 + per);
        d.v0 = uint32_t(t0);
        d.v1 = uint32_t(t1);
        out.push_back(d);
        t0 = t1;
    }
    p.align = std::max<int64_t>(p.align, (ald || ast) ? 16 : es);
    p.transpose_rows = std::max(p.transpose_rows, uint32_t(tr));
}

int64_t auto_chunk_bytes(int64_t bytes_read) {
    // Enough chunks to fill 256 CUs many times over, 4 KiB .. 16 KiB each;
    // past 64 GiB, larger chunks keep the table within a quarter of the
    // chunk limit.
    int64_t c = 4096;
    while (c < 16384 && bytes_read / (2 * c) >= 4096) c *= 2;
    while (bytes_read / c > int64_t(kMaxDescs / 4)) c *= 2;
    return c;
}

// Row-gather lowering of one group (see desc.h).  Returns false, emitting
// nothing, when the group does not qualify; its tasks then take the
// per-task path.
bool lower_gather_group(Plan &p, const std::vector<size_t> &group, int64_t chunk_bytes, std::vector<Desc> &out) {
    const int nd = p.ndim;
    const int64_t es = p.es;
    if (nd < 1 || group.size() < 2 || group.size() > kMaxSegs) return false;
    std::vector<size_t> g(group);
    std::sort(g.begin(), g.end(), [&](size_t a, size_t b) { return p.tasks[a].lo[nd - 1] < p.tasks[b].lo[nd - 1]; });
    const UnitTask &t0 = p.tasks[g[0]];
    const int64_t fan_off = p.dst.shard_devs_off[t0.dst_shard];
    const int64_t nfan = p.dst.shard_devs_off[t0.dst_shard + 1] - fan_off;
    const int32_t rcv0 = p.dst.shard_devs[fan_off];
    // destination local layout
    std::vector<int64_t> ext_d(nd), str_d(nd), dlo(nd);
    for (int d = 0; d < nd; ++d) {
        const int64_t jd = p.dst.dev_shard[int64_t(rcv0) * nd + d];
        dlo[d] = p.dst.bounds[d][jd];
        ext_d[d] = p.dst.bounds[d][jd + 1] - dlo[d];
    }
    for (int d = nd - 1; d >= 0; --d) str_d[d] = d == nd - 1 ? es : str_d[d + 1] * ext_d[d + 1];
    // the segments must tile the destination row with equal, 16-byte widths
    const int64_t wcol = t0.hi[nd - 1] - t0.lo[nd - 1];
    int64_t at = dlo[nd - 1];
    for (size_t k : g) {
        const UnitTask &t = p.tasks[k];
        if (t.lo[nd - 1] != at || t.hi[nd - 1] - t.lo[nd - 1] != wcol) return false;
        at = t.hi[nd - 1];
    }
    if (at != dlo[nd - 1] + ext_d[nd - 1]) return false;
    const int64_t seg_bytes = wcol * es, row_bytes = ext_d[nd - 1] * es;
    if (seg_bytes % 16 || row_bytes % 16) return false;
    // outer levels: drop unit extents, merge dims contiguous on the
    // destination and on every sender
    const size_t ns = g.size();
    std::vector<std::vector<int64_t>> str_s(ns, std::vector<int64_t>(nd)), slo(ns, std::vector<int64_t>(nd));
    for (size_t k = 0; k < ns; ++k) {
        const UnitTask &t = p.tasks[g[k]];
        std::vector<int64_t> ext_s(nd);
        for (int d = 0; d < nd; ++d) {
            const int64_t js = p.src.dev_shard[int64_t(t.sender) * nd + d];
            slo[k][d] = p.src.bounds[d][js];
            ext_s[d] = p.src.bounds[d][js + 1] - slo[k][d];
        }
        for (int d = nd - 1; d >= 0; --d) str_s[k][d] = d == nd - 1 ? es : str_s[k][d + 1] * ext_s[d + 1];
    }
    struct GLevel {
        int64_t n, ds;
        std::vector<int64_t> ss;
    };
    std::vector<GLevel> lv;  // innermost first while building
    for (int d = nd - 2; d >= 0; --d) {
        const int64_t n = t0.hi[d] - t0.lo[d];
        if (n == 1) continue;
        bool merge = !lv.empty() && str_d[d] == lv.back().n * lv.back().ds;
        for (size_t k = 0; k < ns && merge; ++k) merge = str_s[k][d] == lv.back().n * lv.back().ss[k];
        if (merge) {
            lv.back().n *= n;
        } else {
            GLevel l{n, str_d[d], std::vector<int64_t>(ns)};
            for (size_t k = 0; k < ns; ++k) l.ss[k] = str_s[k][d];
            lv.push_back(l);
        }
    }
    if (lv.size() > 3) return false;
    for (const auto &l : lv) {
        if (l.ds % 16) return false;
        for (int64_t x : l.ss)
            if (x % 16) return false;
    }
    uint64_t rows = 1;
    for (const auto &l : lv) rows *= uint64_t(l.n);
    const uint64_t spr = uint64_t(row_bytes / 16), sps = uint64_t(seg_bytes / 16);
    if (rows * spr >= (uint64_t(1) << 31)) return false;
    // per-segment source origin and span (relative offsets stay below 2^32)
    std::vector<Seg> seg(ns);
    for (size_t k = 0; k < ns; ++k) {
        const UnitTask &t = p.tasks[g[k]];
        uint64_t so = 0, span = uint64_t(seg_bytes);
        for (int d = 0; d < nd; ++d) so += uint64_t((t.lo[d] - slo[k][d]) * str_s[k][d]);
        if (so % 16) return false;
        for (const auto &l : lv) span += uint64_t(l.n - 1) * uint64_t(l.ss[k]);
        if (span >= (uint64_t(1) << 32)) return false;
        seg[k].src_base = so;
        seg[k].buf = uint32_t(t.sender);
        for (size_t i = 0; i < lv.size(); ++i) seg[k].ss[i] = uint32_t(uint64_t(lv[i].ss[k]));
    }
    uint64_t dso = 0;
    for (int d = 0; d < nd - 1; ++d) dso += uint64_t((t0.lo[d] - dlo[d]) * str_d[d]);
    const int levels = std::max<int>(1, int(lv.size()));
    Desc d{};
    for (size_t i = 0; i < lv.size(); ++i) d.ds[i] = uint32_t(uint64_t(lv[i].ds));
    d.vpr = uint32_t(spr);
    d.n1 = lv.size() >= 2 ? uint32_t(lv[0].n) : 1u;
    d.n2 = lv.size() >= 3 ? uint32_t(lv[1].n) : 1u;
    const FastDiv f0 = make_fastdiv(d.vpr), f1 = make_fastdiv(d.n1), f2 = make_fastdiv(d.n2),
                  fs = make_fastdiv(uint32_t(sps));
    d.mul_vpr = f0.mul; d.sh_vpr = uint8_t(f0.shift);
    d.mul_n1 = f1.mul;  d.sh_n1 = uint8_t(f1.shift);
    d.mul_n2 = f2.mul;  d.sh_n2 = uint8_t(f2.shift);
    d.run = uint32_t(sps);
    d.batch = fs.mul;
    d.pad[2] = fs.shift;
    d.kind = uint8_t(make_kind(4, uint32_t(levels)));
    d.nfan = uint16_t(nfan);
    d.fan_off = uint32_t(fan_off);
    // Column bands of `band` segments, one after another; each band's chunks
    // are ranges of its slots over consecutive rows.
    const uint64_t band = p.tuning.gather_band > 0 && uint64_t(p.tuning.gather_band) < ns
                              ? uint64_t(p.tuning.gather_band) : uint64_t(ns);
    const uint64_t cv = uint64_t(std::max<int64_t>(16, chunk_bytes / 16)) / 16 * 16;
    uint64_t nchunks = 0;
    for (uint64_t b0 = 0; b0 < ns; b0 += band)
        nchunks += (rows * std::min<uint64_t>(band, ns - b0) * sps + cv - 1) / cv;
    if (p.descs.size() + out.size() + nchunks > kMaxDescs) {
        p.too_many = true;
        return false;
    }
    std::vector<Desc> mine;
    for (uint64_t b0 = 0; b0 < ns; b0 += band) {
        const uint64_t nb = std::min<uint64_t>(band, ns - b0), bw = nb * sps;
        const uint64_t bso = dso + b0 * sps * 16;  // destination offset of the band's first slot
        const FastDiv fb = make_fastdiv(uint32_t(bw));
        d.vpr = uint32_t(bw);
        d.mul_vpr = fb.mul;
        d.sh_vpr = uint8_t(fb.shift);
        d.pad[0] = uint32_t(p.segs.size() + b0);
        d.pad[1] = uint32_t(nb);
        // destination offset of slot v of the band (64-bit), levels innermost first
        auto dst_off = [&](uint64_t v) {
            uint64_t row = v / bw, off = bso + (v - row * bw) * 16;
            for (size_t i = 0; i < lv.size(); ++i) {
                const uint64_t n = uint64_t(lv[i].n);
                const uint64_t idx = i + 1 == lv.size() ? row : row % n;
                off += idx * uint64_t(lv[i].ds);
                row = i + 1 == lv.size() ? 0 : row / n;
            }
            return off;
        };
        const uint64_t total = rows * bw;
        for (uint64_t v0 = 0; v0 < total;) {
            uint64_t v1 = std::min(total, v0 + cv);
            const uint64_t first = dst_off(v0);
            while (dst_off(v1 - 1) + 16 - first >= kMaxChunkSpan) v1 = v0 + (v1 - v0) / 2;
            d.v0 = uint32_t(v0);
            d.v1 = uint32_t(v1);
            d.dst_base = first;
            d.dst_rel0 = uint32_t(first - bso);
            mine.push_back(d);
            v0 = v1;
        }
    }
    p.segs.insert(p.segs.end(), seg.begin(), seg.end());
    out.insert(out.end(), mine.begin(), mine.end());
    p.align = std::max<int64_t>(p.align, 16);
    p.max_fanout = std::max(p.max_fanout, nfan);
    p.gather_fanout = std::max(p.gather_fanout, nfan);
    return true;
}

// Cut each of the last k row-gather chunks (the ones dispatched last) in
// two halves of whole 16-slot groups, so the launch's tail drains in
// shorter pieces.  The second half's origin comes from the kernel's own
// slot -> offset arithmetic on the descriptor, so dst_base and dst_rel0 stay
// the offsets of each chunk's first slot.
void halve_gather_tail(std::vector<Desc> &g, size_t k) {
    k = std::min(k, g.size());
    std::vector<Desc> out;
    out.reserve(2 * k);
    for (size_t i = g.size() - k; i < g.size(); ++i) {
        const Desc &d = g[i];
        const uint32_t h = (d.v1 - d.v0) / 2 / 16 * 16;
        if (h == 0) {
            out.push_back(d);
            continue;
        }
        Desc a = d, b = d;
        a.v1 = b.v0 = d.v0 + h;
        const uint32_t row = fastdiv(b.v0, d.mul_vpr, d.sh_vpr), j = b.v0 - row * d.vpr;
        uint32_t i1 = 0, i2 = 0, i3 = 0;
        switch (kind_levels(d.kind)) {
            case 1: row_indices<1>(d, row, i1, i2, i3); break;
            case 2: row_indices<2>(d, row, i1, i2, i3); break;
            default: row_indices<3>(d, row, i1, i2, i3); break;
        }
        const uint32_t rel = i1 * d.ds[0] + i2 * d.ds[1] + i3 * d.ds[2] + 16u * j;
        b.dst_base = d.dst_base + uint64_t(rel - d.dst_rel0);
        b.dst_rel0 = rel;
        out.push_back(a);
        out.push_back(b);
    }
    g.resize(g.size() - k);
    g.insert(g.end(), out.begin(), out.end());
}

#ifndef RS_UG_MIN_RUN
#define RS_UG_MIN_RUN 2048u
#endif
#ifndef RS_UNIT_MAX_FAN
#define RS_UNIT_MAX_FAN 1  // largest receiver count the unit gather takes
#endif
#ifndef RS_UNIT_MAX_SEG
#define RS_UNIT_MAX_SEG 2048  // the unit gather takes mean segment widths below this (bytes)
#endif

// Unaligned row gather of one group (see desc.h): segments of any widths
// tiling the destination row (one segment per row too, when its rows are in
// different 16-byte phases on the two sides), destination rows contiguous
// whole or in runs.  Returns false, emitting nothing, when the group does
// not qualify.
bool lower_gather_unaligned(Plan &p, const std::vector<size_t> &group, int64_t chunk_bytes, std::vector<Desc> &out,
                            std::vector<Desc> &unit_out) {
    const int nd = p.ndim;
    const int64_t es = p.es;
    if (nd < 1 || group.empty() || group.size() > kMaxSegs) return false;
    std::vector<size_t> g(group);
    std::sort(g.begin(), g.end(), [&](size_t a, size_t b) { return p.tasks[a].lo[nd - 1] < p.tasks[b].lo[nd - 1]; });
    const UnitTask &t0 = p.tasks[g[0]];
    const int64_t fan_off = p.dst.shard_devs_off[t0.dst_shard];
    const int64_t nfan = p.dst.shard_devs_off[t0.dst_shard + 1] - fan_off;
    const int32_t rcv0 = p.dst.shard_devs[fan_off];
    std::vector<int64_t> ext_d(nd), str_d(nd), dlo(nd);
    for (int d = 0; d < nd; ++d) {
        const int64_t jd = p.dst.dev_shard[int64_t(rcv0) * nd + d];
        dlo[d] = p.dst.bounds[d][jd];
        ext_d[d] = p.dst.bounds[d][jd + 1] - dlo[d];
    }
    for (int d = nd - 1; d >= 0; --d) str_d[d] = d == nd - 1 ? es : str_d[d + 1] * ext_d[d + 1];
    // the segments tile the destination row (segments shorter than 16 bytes
    // make some slots hold more than two pieces: the kernel's rare path)
    int64_t at = dlo[nd - 1];
    for (size_t k : g) {
        const UnitTask &t = p.tasks[k];
        if (t.lo[nd - 1] != at) return false;
        at = t.hi[nd - 1];
    }
    if (at != dlo[nd - 1] + ext_d[nd - 1]) return false;
    const int64_t row_bytes = ext_d[nd - 1] * es;
    if (row_bytes >= (int64_t(1) << 31)) return false;
    // destination rows: contiguous across the inner outer dimensions up to
    // the first one that does not span its whole dimension; the dimensions
    // from that one outward cut the group into runs of contiguous rows (one
    // run when every inner extent is whole).  Row r of the group is its
    // C-order index over the outer dimensions, so run k holds rows
    // [k * run_rows, (k + 1) * run_rows).
    int64_t acc = row_bytes;
    uint64_t rows = 1, run_rows = 1;
    int brk = -1;
    for (int d = nd - 2; d >= 0; --d) {
        const int64_t n = t0.hi[d] - t0.lo[d];
        rows *= uint64_t(n);
        if (n == 1 || brk >= 0) continue;
        if (str_d[d] == acc) {
            acc *= n;
            run_rows *= uint64_t(n);
        } else {
            brk = d;
        }
    }
    if (rows >= (uint64_t(1) << 31)) return false;
    // source levels: drop unit extents, merge dims contiguous on every sender
    const size_t ns = g.size();
    std::vector<std::vector<int64_t>> str_s(ns, std::vector<int64_t>(nd)), slo(ns, std::vector<int64_t>(nd));
    for (size_t k = 0; k < ns; ++k) {
        const UnitTask &t = p.tasks[g[k]];
        std::vector<int64_t> ext_s(nd);
        for (int d = 0; d < nd; ++d) {
            const int64_t js = p.src.dev_shard[int64_t(t.sender) * nd + d];
            slo[k][d] = p.src.bounds[d][js];
            ext_s[d] = p.src.bounds[d][js + 1] - slo[k][d];
        }
        for (int d = nd - 1; d >= 0; --d) str_s[k][d] = d == nd - 1 ? es : str_s[k][d + 1] * ext_s[d + 1];
    }
    struct SLevel {
        int64_t n;
        std::vector<int64_t> ss;
    };
    std::vector<SLevel> lv;  // innermost first
    for (int d = nd - 2; d >= 0; --d) {
        const int64_t n = t0.hi[d] - t0.lo[d];
        if (n == 1) continue;
        bool merge = !lv.empty();
        for (size_t k = 0; k < ns && merge; ++k) merge = str_s[k][d] == lv.back().n * lv.back().ss[k];
        if (merge) {
            lv.back().n *= n;
        } else {
            SLevel l{n, std::vector<int64_t>(ns)};
            for (size_t k = 0; k < ns; ++k) l.ss[k] = str_s[k][d];
            lv.push_back(l);
        }
    }
    if (lv.size() > 3) return false;
    std::vector<Seg> seg(ns);
    for (size_t k = 0; k < ns; ++k) {
        const UnitTask &t = p.tasks[g[k]];
        uint64_t so = 0, span = uint64_t((t.hi[nd - 1] - t.lo[nd - 1]) * es);
        for (int d = 0; d < nd; ++d) so += uint64_t((t.lo[d] - slo[k][d]) * str_s[k][d]);
        for (const auto &l : lv) span += uint64_t(l.n - 1) * uint64_t(l.ss[k]);
        if (span >= (uint64_t(1) << 32)) return false;
        seg[k] = Seg{so, {0u, 0u, 0u}, uint32_t(t.sender), uint32_t((t.lo[nd - 1] - dlo[nd - 1]) * es), 0u};
        for (size_t i = 0; i < lv.size(); ++i) seg[k].ss[i] = uint32_t(uint64_t(lv[i].ss[k]));
    }
    uint64_t d0 = 0;  // the group's first byte in the receivers' buffers
    for (int d = 0; d < nd - 1; ++d) d0 += uint64_t((t0.lo[d] - dlo[d]) * str_d[d]);
    if (ns == 1) {
        // One sender per row: only where the per-task lowering would need the
        // realignment kernel (the two sides' rows in different 16-byte
        // phases); slots of the contiguous destination rows then keep every
        // cache line within one workgroup.
        bool same_phase = row_bytes % 16 == 0 && (seg[0].src_base - d0) % 16 == 0;
        for (const auto &l : lv) same_phase = same_phase && l.ss[0] % 16 == 0;
        for (int d = 0; d <= brk; ++d) same_phase = same_phase && str_d[d] % 16 == 0;
        if (same_phase) return false;
    }
    const uint64_t run_bytes = run_rows * uint64_t(row_bytes);
    const int levels = std::max<int>(1, int(lv.size()));
    Desc d{};
    d.vpr = uint32_t(row_bytes);
    d.n1 = lv.size() >= 2 ? uint32_t(lv[0].n) : 1u;
    d.n2 = lv.size() >= 3 ? uint32_t(lv[1].n) : 1u;
    const uint32_t wnom = uint32_t(row_bytes / int64_t(ns));
    const FastDiv f0 = make_fastdiv(d.vpr), f1 = make_fastdiv(d.n1), f2 = make_fastdiv(d.n2), fw = make_fastdiv(wnom);
    d.mul_vpr = f0.mul; d.sh_vpr = uint8_t(f0.shift);
    d.mul_n1 = f1.mul;  d.sh_n1 = uint8_t(f1.shift);
    d.mul_n2 = f2.mul;  d.sh_n2 = uint8_t(f2.shift);
    d.run = wnom;
    d.batch = fw.mul;
    d.pad[2] = fw.shift;
    d.kind = uint8_t(make_kind(4, uint32_t(levels)));
    d.nfan = uint16_t(nfan);
    d.fan_off = uint32_t(fan_off);
    d.pad[0] = uint32_t(p.segs.size());
    d.pad[1] = uint32_t(ns);
    const uint64_t cv = uint64_t(std::max<int64_t>(16, chunk_bytes / 16)) / 16 * 16;
    // each run is chunked on its own: runs shorter than RS_UG_MIN_RUN bytes
    // (which would make very short chunks) stay with the per-task lowering
    if (brk >= 0 && (run_bytes < std::min<uint64_t>(16 * cv, RS_UG_MIN_RUN) || rows / run_rows > kMaxDescs / 4))
        return false;
    // run starts in the receivers' buffers, C order over dimensions 0..brk
    std::vector<uint64_t> run_d0(1, d0);
    for (int d = 0; d <= brk; ++d) {
        const int64_t n = t0.hi[d] - t0.lo[d];
        std::vector<uint64_t> next;
        next.reserve(run_d0.size() * uint64_t(n));
        for (uint64_t b : run_d0)
            for (int64_t i = 0; i < n; ++i) next.push_back(b + uint64_t(i * str_d[d]));
        run_d0.swap(next);
    }
    uint64_t nchunks = 0;
    for (uint64_t b : run_d0) nchunks += ((b + run_bytes + 15) / 16 - b / 16 + cv - 1) / cv;
    if (p.descs.size() + out.size() + nchunks > kMaxDescs) {
        p.too_many = true;
        return false;
    }
    std::vector<Desc> mine;
    // One receiver and segments under RS_UNIT_MAX_SEG bytes on average: the
    // unit gather (unaligned loads and stores, see desc.h; a segment under
    // 16 bytes is one unit moved byte by byte).
    // The slot form spends its time on slots that straddle two segments
    // (or rows), which short segments make frequent.  Measured against
    // destination slots: 8 % faster with 770-byte segments at fan-out 1, 18 %
    // with 4-byte segments among them; slower at fan-out 2 and with rows of
    // 6 KiB and more from one sender.
    bool unit = nfan <= int64_t(RS_UNIT_MAX_FAN) && row_bytes < int64_t(RS_UNIT_MAX_SEG) * int64_t(ns);
    uint32_t upr = 0;  // units per row
    bool unit_short = false;
    for (size_t k = 0; k < ns; ++k) {
        const uint32_t w = (k + 1 < ns ? seg[k + 1].col : uint32_t(row_bytes)) - seg[k].col;
        unit_short = unit_short || w < 16;
        seg[k].pad = upr;
        upr += (w + 15) / 16;
    }
    if (unit) {
        const uint64_t total = run_rows * upr;
        if (total >= (uint64_t(1) << 32)) unit = false;
    }
    if (unit) {
        const uint64_t total = run_rows * upr;
        const uint64_t per = (total + cv - 1) / cv;
        if (p.descs.size() + out.size() + unit_out.size() + per * run_d0.size() > kMaxDescs) {
            p.too_many = true;
            return false;
        }
        Desc u = d;
        u.kind = uint8_t(make_kind(4, uint32_t(levels)) | kUnitGather);
        u.ds[0] = unit_short ? kUShortSegs : 0u;
        u.vpr = upr;
        const FastDiv fu = make_fastdiv(upr), fn = make_fastdiv(std::max<uint32_t>(1, upr / uint32_t(ns)));
        u.mul_vpr = fu.mul;
        u.sh_vpr = uint8_t(fu.shift);
        u.batch = fn.mul;
        u.pad[2] = fn.shift;
        u.run = uint32_t(row_bytes);
        for (size_t k = 0; k < run_d0.size(); ++k) {
            for (uint64_t v0 = 0; v0 < total; v0 += cv) {
                const uint64_t r_first = v0 / upr;
                u.v0 = uint32_t(v0);
                u.v1 = uint32_t(std::min(total, v0 + cv));
                u.ss[0] = uint32_t(uint64_t(k) * run_rows);
                u.ss[1] = uint32_t(r_first);
                u.ss[2] = 0;
                u.src_rel0 = 0;
                u.dst_base = run_d0[k] + r_first * uint64_t(row_bytes);
                mine.push_back(u);
            }
        }
    }
    if (!unit) {
        mine.reserve(nchunks);
        for (size_t k = 0; k < ns; ++k)
            if ((k + 1 < ns ? seg[k + 1].col : uint32_t(row_bytes)) - seg[k].col < 16u) d.ds[0] = kUShortSegs;
    }
    for (size_t k = 0; k < run_d0.size() && !unit; ++k) {
        const uint64_t rd0 = run_d0[k];  // this run's first byte
        const uint64_t s_first = rd0 / 16, s_end = (rd0 + run_bytes + 15) / 16;
        for (uint64_t s0 = s_first; s0 < s_end; s0 += cv) {
            const uint64_t nsl = std::min(cv, s_end - s0), base = 16 * s0;
            d.v0 = 0;
            d.v1 = uint32_t(nsl);
            d.dst_base = base;
            uint64_t row0 = uint64_t(k) * run_rows;
            int64_t cofs0;
            if (base <= rd0) {
                cofs0 = int64_t(base) - int64_t(rd0);  // in (-16, 0]
            } else {
                const uint64_t q = base - rd0, dr = q / uint64_t(row_bytes);
                row0 += dr;
                cofs0 = int64_t(q - dr * uint64_t(row_bytes));
            }
            d.ss[0] = uint32_t(row0);
            d.ss[1] = uint32_t(cofs0);
            d.ss[2] = uint32_t(base < rd0 ? rd0 - base : 0);
            d.src_rel0 = uint32_t(std::min<uint64_t>(16 * nsl, rd0 + run_bytes - base));
            mine.push_back(d);
            p.gather_u_bytes += d.src_rel0 - d.ss[2];
            p.gather_u_room += 16 * cv;
        }
    }
    p.segs.insert(p.segs.end(), seg.begin(), seg.end());
    (unit ? unit_out : out).insert((unit ? unit_out : out).end(), mine.begin(), mine.end());
    p.align = std::max<int64_t>(p.align, 16);
    p.max_fanout = std::max(p.max_fanout, nfan);
    if (unit) {
        p.unit_fanout = std::max(p.unit_fanout, nfan);
        p.unit_segs = std::max(p.unit_segs, int64_t(ns));
    } else {
        p.gather_u_fanout = std::max(p.gather_u_fanout, nfan);
        p.gather_u_segs = std::max(p.gather_u_segs, int64_t(ns));
        p.gather_u_short = p.gather_u_short || (d.ds[0] & kUShortSegs) != 0;
    }
    return true;
}

}  // namespace

void lower(Plan &p) {
    const int nd = p.ndim;
    const int64_t es = p.es;
    p.descs.clear();
    p.fan.assign(p.dst.shard_devs.begin(), p.dst.shard_devs.end());
    p.align = 1;
    p.lds_bytes = 0;
    p.transpose_rows = 0;
    p.too_many = false;
    p.tile_span_too_long = false;
    p.max_fanout = 0;
    p.bytes_read = 0;
    for (const auto &t : p.tasks) p.bytes_read += t.bytes;
    const int64_t chunk = p.tuning.chunk_bytes > 0 ? p.tuning.chunk_bytes : auto_chunk_bytes(p.bytes_read);

    // Row groups: tasks sharing the receiver set and the box in every
    // dimension but the last (0x100: RESHARD_NO_GATHER; strategies copy per task).
    p.segs.clear();
    p.gather_fanout = 0;
    p.gather_u_fanout = 0;
    p.gather_u_segs = 0;
    p.gather_u_bytes = 0;
    p.gather_u_room = 0;
    p.gather_u_short = false;
    p.unit_fanout = 0;
    p.unit_segs = 0;
    std::vector<Desc> gdescs, udescs, unitdescs;
    std::vector<char> handled(p.tasks.size(), 0);
    bool permuted = false;
    for (int k = 0; k < nd; ++k)
        permuted = permuted || (!p.sperm.empty() && p.sperm[size_t(k)] != k) ||
                   (!p.dperm.empty() && p.dperm[size_t(k)] != k);
    std::vector<Desc> tdescs;
    if (!(p.flags & 0x100u) && !(p.flags & 0x60u) && !permuted) {
        std::map<std::vector<int64_t>, std::vector<size_t>> groups;
        for (size_t i = 0; i < p.tasks.size(); ++i) {
            const UnitTask &t = p.tasks[i];
            std::vector<int64_t> key{t.dst_shard};
            for (int d = 0; d + 1 < nd; ++d) {
                key.push_back(t.lo[d]);
                key.push_back(t.hi[d]);
            }
            groups[key].push_back(i);
        }
        for (const auto &kv : groups)
            if (lower_gather_group(p, kv.second, chunk, gdescs) ||
                lower_gather_unaligned(p, kv.second, chunk, udescs, unitdescs))
                for (size_t i : kv.second) handled[i] = 1;
        // With automatic chunk sizes, the last fifth of the row-gather chunks
        // in halves (same machine, interleaved: workload 5 360.8 -> 358.6 us,
        // workload 3 545.8 -> 539.7 us, within 0.4 % for the last sixth to
        // the last third; quarters were slower, 362.3 and 561.4 us).
        if (p.tuning.chunk_bytes <= 0) halve_gather_tail(gdescs, gdescs.size() / 5);
    }

    std::vector<int64_t> ext_s(nd), ext_d(nd), str_s(nd), str_d(nd);
    for (size_t ti = 0; ti < p.tasks.size(); ++ti) {
        if (p.too_many || p.tile_span_too_long) break;  // the plan fails: stop lowering
        if (handled[ti]) continue;
        const auto &t = p.tasks[ti];
        const int64_t fan_off = p.dst.shard_devs_off[t.dst_shard];
        const int64_t nfan = p.dst.shard_devs_off[t.dst_shard + 1] - fan_off;
        p.max_fanout = std::max(p.max_fanout, nfan);
        const int32_t rcv0 = p.dst.shard_devs[fan_off];
        // local boxes of the sender and of (any) receiver
        uint64_t so = 0, dso = 0;
        for (int d = 0; d < nd; ++d) {
            const int64_t js = p.src.dev_shard[int64_t(t.sender) * nd + d];
            const int64_t jd = p.dst.dev_shard[int64_t(rcv0) * nd + d];
            ext_s[d] = p.src.bounds[d][js + 1] - p.src.bounds[d][js];
            ext_d[d] = p.dst.bounds[d][jd + 1] - p.dst.bounds[d][jd];
        }
        // byte stride of each tensor dimension in the (possibly permuted)
        // dense buffers: buffer dimension k is tensor dimension perm[k]
        int64_t a = es, b = es;
        for (int k = nd - 1; k >= 0; --k) {
            const int ds_ = p.sperm.empty() ? k : p.sperm[size_t(k)];
            const int dd_ = p.dperm.empty() ? k : p.dperm[size_t(k)];
            str_s[ds_] = a;
            str_d[dd_] = b;
            a *= ext_s[ds_];
            b *= ext_d[dd_];
        }
        for (int d = 0; d < nd; ++d) {
            const int64_t js = p.src.dev_shard[int64_t(t.sender) * nd + d];
            const int64_t jd = p.dst.dev_shard[int64_t(rcv0) * nd + d];
            so += uint64_t((t.lo[d] - p.src.bounds[d][js]) * str_s[d]);
            dso += uint64_t((t.lo[d] - p.dst.bounds[d][jd]) * str_d[d]);
        }
        // collapse, in the receivers' dimension order: drop unit extents,
        // merge dims contiguous on both sides
        std::vector<Level> g;  // innermost first while building
        for (int k = nd - 1; k >= 0; --k) {
            const int d = p.dperm.empty() ? k : p.dperm[size_t(k)];
            const int64_t n = t.hi[d] - t.lo[d];
            if (n == 1) continue;
            if (!g.empty() && str_s[d] == g.back().n * g.back().ss && str_d[d] == g.back().n * g.back().ds)
                g.back().n *= n;
            else
                g.push_back({n, str_s[d], str_d[d]});
        }
        // Contiguous along different dimensions on the two sides (a
        // permuted layout): tiles transposed through LDS.
        if (!g.empty() && g.front().ds == es && g.front().ss != es) {
            size_t ia = 0;
            for (size_t i = 1; i < g.size(); ++i)
                if (g[i].ss == es) ia = i;
            const int64_t te = int64_t(tile_elems(uint32_t(es)));
            if (ia > 0 && te * g.front().ss < (int64_t(1) << 31) && te * g[ia].ds < (int64_t(1) << 31)) {
                TPiece tp{so, dso, g[ia].n, g.front().n, g.front().ss, g[ia].ds, {}};
                for (size_t i = g.size(); i-- > 1;)
                    if (i != ia) tp.outer.push_back(g[i]);  // outermost first
                emit_transpose(p, tp, t.sender, fan_off, nfan, chunk, tdescs);
                continue;
            }
        }
        int64_t run = es;
        if (!g.empty() && g.front().ss == es && g.front().ds == es) {
            run = g.front().n * es;
            g.erase(g.begin());
        }
        std::reverse(g.begin(), g.end());  // outermost first

        // Head / body / tail split so the body moves whole 16-byte vectors
        // when both sides share the 16-byte phase on every row.
        bool phase_ok = ((so - dso) % 16) == 0;
        for (const auto &l : g) phase_ok = phase_ok && (l.ss % 16 == 0) && (l.ds % 16 == 0);
        std::vector<Piece> parts;
        if (phase_ok && run >= 32) {
            const int64_t head = std::min<int64_t>(run, int64_t((16 - so % 16) % 16));
            const int64_t body = (run - head) / 16 * 16;
            const int64_t tail = run - head - body;
            int64_t at = 0;
            for (int64_t len : {head, body, tail}) {
                if (len > 0) {
                    Piece pc{so + uint64_t(at), dso + uint64_t(at), len, g, 1};
                    pc.w = pick_width(pc.src_off, pc.dst_off, pc.run, pc.outer);
                    parts.push_back(pc);
                }
                at += len;
            }
        } else if (run >= kRealignMinRun && !(p.flags & 0x8u) && !(p.flags & 0x60u)) {
            // (0x8: RESHARD_NO_REALIGN; 0x60: a comparison strategy, direct chunks only)
            // different 16-byte phases: stage rows through LDS, segments of
            // at most kRealignSeg bytes
            for (int64_t at = 0; at < run; at += kRealignSeg) {
                Piece pc{so + uint64_t(at), dso + uint64_t(at), std::min(kRealignSeg, run - at), g, 16};
                pc.realign = true;
                parts.push_back(pc);
            }
        } else {
            Piece pc{so, dso, run, g, 1};
            pc.w = pick_width(so, dso, run, g);
            parts.push_back(pc);
        }
        for (const auto &pc : parts) split_emit(p, pc, t.sender, fan_off, nfan, chunk);
    }
    if (p.too_many || p.tile_span_too_long) return;  // the plan fails: nothing to order
    if (!(p.flags & 0x4u)) {
        // destination-major chunk order: receiver set, then the byte offset
        // of the chunk's first vector in the receivers' buffers
        std::vector<std::pair<std::pair<uint32_t, uint64_t>, size_t>> key(p.descs.size());
        for (size_t i = 0; i < p.descs.size(); ++i) key[i] = {{p.descs[i].fan_off, p.descs[i].dst_base}, i};
        std::stable_sort(key.begin(), key.end(),
                         [](const auto &a, const auto &b) { return a.first < b.first; });
        std::vector<Desc> sorted(p.descs.size());
        for (size_t i = 0; i < key.size(); ++i) sorted[i] = p.descs[key[i].second];
        p.descs.swap(sorted);
    }
    // direct chunks first, then row-gather chunks, realignment chunks last
    // (three kernels)
    std::stable_partition(p.descs.begin(), p.descs.end(), [](const Desc &d) { return !kind_realign(d.kind); });
    p.n_direct = 0;
    while (p.n_direct < p.descs.size() && !kind_realign(p.descs[p.n_direct].kind)) ++p.n_direct;
    p.descs.insert(p.descs.begin() + std::ptrdiff_t(p.n_direct), gdescs.begin(), gdescs.end());
    p.n_gather = gdescs.size();
    udescs.insert(udescs.end(), unitdescs.begin(), unitdescs.end());  // unit chunks last in the section
    p.descs.insert(p.descs.begin() + std::ptrdiff_t(p.n_direct + p.n_gather), udescs.begin(), udescs.end());
    p.n_gather_u = udescs.size();
    p.n_unit = unitdescs.size();
    if (!(p.flags & 0x4u)) {
        // tile chunks in destination order too (receiver set, then the
        // destination offset of the chunk's first tile), so the tiles
        // resident together write neighbouring destination bytes whichever
        // sender they read (same machine, interleaved: transposed workload 5
        // 382.5 -> 372.3 us, fp32 385.6 -> 379.8, one replica 150.8 ->
        // 147.4, source side permuted 409.5 -> 406.6; task order before)
        std::vector<std::pair<std::pair<uint32_t, uint64_t>, size_t>> key(tdescs.size());
        for (size_t i = 0; i < tdescs.size(); ++i) {
            const Desc &d = tdescs[i];
            key[i] = {{d.fan_off, d.dst_base + uint64_t(tile_offsets(d, d.v0, uint32_t(p.es)).dst)}, i};
        }
        std::stable_sort(key.begin(), key.end(), [](const auto &a, const auto &b) { return a.first < b.first; });
        std::vector<Desc> sorted(tdescs.size());
        for (size_t i = 0; i < key.size(); ++i) sorted[i] = tdescs[key[i].second];
        tdescs.swap(sorted);
    }
    p.descs.insert(p.descs.begin() + std::ptrdiff_t(p.n_direct + p.n_gather + p.n_gather_u), tdescs.begin(),
                   tdescs.end());
    p.n_transpose = tdescs.size();
    if (p.descs.size() > kMaxDescs) p.too_many = true;
    p.n_phase1 = p.n_direct;
    if (p.flags & 0x20u) {
        // Send/recv analogue (Section 3.1): the sender's slice is read once
        // per receiver -- every chunk becomes one fan-out-1 chunk per receiver.
        std::vector<Desc> out;
        out.reserve(p.descs.size() * size_t(std::max<int64_t>(1, p.max_fanout)));
        for (const Desc &d : p.descs)
            for (uint32_t k = 0; k < d.nfan; ++k) {
                Desc e = d;
                e.fan_off = d.fan_off + k;
                e.nfan = 1;
                out.push_back(e);
            }
        p.descs.swap(out);
        p.n_direct = p.n_phase1 = p.descs.size();
        p.bytes_read = 0;
        for (const auto &t : p.tasks)
            p.bytes_read += t.bytes * (p.dst.shard_devs_off[t.dst_shard + 1] - p.dst.shard_devs_off[t.dst_shard]);
    } else if (p.flags & 0x40u) {
        // Send/recv + all-gather analogue (Section 3.1): phase 1 hands the
        // slice's chunks round-robin to its receivers (each part read once
        // from the sender); phase 2 has every receiver pull the parts it
        // lacks from the receiver that holds them (a second launch).
        std::vector<Desc> ph1, ph2;
        uint64_t c = 0;
        for (const Desc &d : p.descs) {
            const uint32_t owner = uint32_t(c++ % d.nfan);
            Desc e = d;
            e.fan_off = d.fan_off + owner;
            e.nfan = 1;
            ph1.push_back(e);
            for (uint32_t k = 0; k < d.nfan; ++k) {
                if (k == owner) continue;
                Desc g = d;  // same offsets: replicas share one local layout
                g.src_buf = uint16_t(p.src.ndev + p.fan[d.fan_off + owner]);
                g.src_base = d.dst_base;
                g.src_rel0 = d.dst_rel0;
                for (int l = 0; l < 3; ++l) g.ss[l] = d.ds[l];
                g.fan_off = d.fan_off + k;
                g.nfan = 1;
                ph2.push_back(g);
            }
        }
        p.n_phase1 = ph1.size();
        ph1.insert(ph1.end(), ph2.begin(), ph2.end());
        p.descs.swap(ph1);
        p.n_direct = p.descs.size();
        p.bytes_read = 0;
        for (const auto &t : p.tasks)
            p.bytes_read += t.bytes * (p.dst.shard_devs_off[t.dst_shard + 1] - p.dst.shard_devs_off[t.dst_shard]);
    }
    p.direct_fanout = 0;
    for (size_t i = 0; i < p.n_direct; ++i) p.direct_fanout = std::max<int64_t>(p.direct_fanout, p.descs[i].nfan);
    p.bytes_written = 0;
    p.dst_local_numel.assign(p.dst.ndev, 0);
    p.src_local_numel.assign(p.src.ndev, 0);
    std::vector<int64_t> shp(nd);
    for (int64_t dev = 0; dev < p.dst.ndev; ++dev) {
        local_shape(p, 1, dev, shp.data());
        int64_t n = 1;
        for (int64_t x : shp) n *= x;
        p.dst_local_numel[dev] = n;
        p.bytes_written += n * es;
    }
    for (int64_t dev = 0; dev < p.src.ndev; ++dev) {
        local_shape(p, 0, dev, shp.data());
        int64_t n = 1;
        for (int64_t x : shp) n *= x;
        p.src_local_numel[dev] = n;
    }
}

void local_shape(const Plan &p, int side, int64_t dev, int64_t *out) {
    const Layout &L = side == 0 ? p.src : p.dst;
    const std::vector<int> &perm = side == 0 ? p.sperm : p.dperm;
    for (int k = 0; k < p.ndim; ++k) {
        const int d = perm.empty() ? k : perm[size_t(k)];
        const int64_t j = L.dev_shard[dev * p.ndim + d];
        out[k] = L.bounds[d][j + 1] - L.bounds[d][j];
    }
}

}  // namespace rs
