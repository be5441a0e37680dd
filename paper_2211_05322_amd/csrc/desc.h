// desc.h -- descriptor table the resharding kernels run from.
//
// One descriptor is one workgroup's chunk of work: a range of W-byte vectors
// inside a "piece", where a piece is part of one unit task's slice seen as
//   (outer level 3) x (outer level 2) x (outer level 1) x (run of vpr vectors)
// with independent byte strides on the sender side and the receiver side.
// The run is contiguous in both buffers.  The sender buffer is read once and
// every receiver gets the same bytes at the same local offset (replicas of a
// destination slice share one local layout).
//
// Addressing: a descriptor carries the 64-bit byte offsets of its chunk's
// first vector (src_base / dst_base).  Offsets inside a piece grow with the
// vector index (dense C-order strides), and the planner keeps every chunk's
// span below 2^32 bytes on both sides, so the offset of any vector relative
// to the chunk's first one is computed exactly in 32-bit modular arithmetic
// from strides taken modulo 2^32.  The kernel thus forms every address as a
// workgroup-uniform 64-bit base plus a 32-bit per-lane offset.
//
// Index arithmetic uses division by invariant integers through a multiply and
// shift (Granlund & Montgomery, "Division by invariant integers using
// multiplication", PLDI 1994, the round-up method for N = 32): for a divisor
// d in [1, 2^31] let l = ceil(log2 d) and m = floor(2^32 (2^l - d) / d) + 1;
// then floor(n / d) = (mulhi(m, n) + n) >> l for every 32-bit n.
// The helpers are constexpr so the same code serves host and device.
#pragma once

#include <stdint.h>

namespace rs {

struct FastDiv {
    uint32_t mul;
    uint32_t shift;
};

constexpr FastDiv make_fastdiv(uint32_t d) {
    uint32_t l = 0;
    while ((uint64_t(1) << l) < d) ++l;
    const uint64_t m = ((uint64_t(1) << 32) * ((uint64_t(1) << l) - d)) / d + 1;
    return FastDiv{uint32_t(m), l};
}

constexpr uint32_t fastdiv(uint32_t n, uint32_t mul, uint32_t shift) {
    const uint64_t t = (uint64_t(mul) * n) >> 32;
    return uint32_t((t + n) >> shift);
}

// Kernel variant: log2 of the vector width, the number of outer levels, and
// whether the chunk takes the LDS realignment path (source and destination
// rows in different 16-byte phases).
constexpr uint32_t kRealign = 0x80u;
constexpr uint32_t make_kind(uint32_t log2w, uint32_t levels) { return log2w | (levels << 4); }
constexpr uint32_t kind_log2w(uint32_t kind) { return kind & 0xFu; }
constexpr uint32_t kind_levels(uint32_t kind) { return (kind >> 4) & 0x7u; }
constexpr bool kind_realign(uint32_t kind) { return (kind & kRealign) != 0; }

// LDS realignment path.  A workgroup stages `batch` rows of a chunk at a
// time: row i of the batch occupies words [i*m, (i+1)*m) of the staging area,
// which starts kRealignFront bytes into LDS; word j of a row holds the
// source's 16-byte aligned word j counted from the one holding the row's
// first byte.  m = words per staged row = (run + 30) / 16 bounds both the
// source words and the 16-byte destination slots a row of `run` bytes can
// touch.  kRealignBack bytes after the last row keep the 5-dword reads of
// the last slot inside the allocation.
constexpr uint32_t kRealignFront = 16;
constexpr uint32_t kRealignBack = 32;
constexpr uint32_t kRealignStageBytes = 16384;  // staged row bytes per pass, at most
constexpr uint32_t realign_words(uint32_t run) { return (run + 30u) / 16u; }
constexpr uint32_t realign_lds_bytes(uint32_t batch, uint32_t m) {
    return kRealignFront + batch * m * 16u + kRealignBack;
}

struct alignas(16) Desc {
    uint64_t src_base;   // byte offset of the chunk's first vector in the sender buffer
    uint64_t dst_base;   // byte offset of the chunk's first vector in every receiver buffer
    uint32_t ss[3];      // sender byte strides of outer levels 1..3 (1 = innermost), mod 2^32
    uint32_t ds[3];      // receiver byte strides of outer levels 1..3, mod 2^32
    uint32_t src_rel0;   // piece-relative sender offset of vector v0, mod 2^32
    uint32_t dst_rel0;   // piece-relative receiver offset of vector v0, mod 2^32
    uint32_t v0, v1;     // this chunk: vectors [v0, v1) of the piece
    uint32_t vpr;        // vectors per run
    uint32_t n1, n2;     // extents of outer levels 1 and 2 (level 3 is bounded by v1)
    uint32_t mul_vpr, mul_n1, mul_n2;  // fast-division multipliers
    uint32_t run;        // realignment path: bytes per row (v0, v1, vpr then count rows / words)
    uint32_t batch;      // realignment path: rows staged in LDS per pass
    uint8_t sh_vpr, sh_n1, sh_n2;      // fast-division shifts
    uint8_t kind;        // make_kind(log2 W, levels) [| kRealign], levels in 1..3
    uint16_t src_buf;    // sender: index into the source pointer table
    uint16_t nfan;       // number of receivers
    uint32_t fan_off;    // receivers: fan[fan_off .. fan_off + nfan) index the dst table
    uint32_t pad[3];
};
static_assert(sizeof(Desc) == 112, "descriptor layout is shared by host and device");

// Row-gather path.  A row group is the set of unit tasks that share one
// receiver set and one box in every dimension but the last, and cut the
// receivers' rows into equal 16-byte-aligned column segments, one per task
// (each from its own sender).  A gather chunk is a range of 16-byte slots of
// whole destination rows; slot j of a row belongs to segment j / sps.  Its
// descriptor uses: vpr = slots per row, run = sps, batch = fast-division
// multiplier of sps and pad[2] its shift, pad[0] = first segment entry,
// pad[1] = number of segments; ds[] and dst_base/dst_rel0 as usual.  ss[],
// src_buf and src_base are unused: every segment entry carries its sender,
// the 64-bit offset of the group's first row at the segment's first column,
// and the sender's strides of the outer levels (mod 2^32).  Source offsets
// are relative to that origin and below 2^32.
//
// Unaligned row gather (own section and kernel).  For row groups whose
// segments tile the destination row in any widths of at least 16 bytes and
// whose destination rows are contiguous (or contiguous in runs, each run its
// own region: its chunks carry its first row in row0), the chunks cover
// 16-byte slots of the destination buffer itself (buffer-aligned, so a slot
// may hold the end of one segment or row and the start of the next: at most
// two pieces).
// Fields: v1 = slots in the chunk (v0 = 0), dst_base = byte offset of its
// first slot; vpr = row bytes with mul_vpr/sh_vpr; n1, n2 and their
// multipliers = the source levels; ss[0] = row0 and ss[1] = cofs0 (int32):
// chunk byte c lies at row row0 + (c + cofs0) / vpr, column (c + cofs0) mod
// vpr; ss[2] = reg_lo, src_rel0 = reg_hi: the chunk bytes [reg_lo, reg_hi)
// belong to the group; run = nominal segment width (vpr / segments, a first
// guess for the segment of a column) with batch/pad[2] its fast division;
// pad[0], pad[1] the segment entries; ds[0] = kUShortSegs when some segment
// is shorter than 16 bytes (a slot may then hold three or more pieces).
// Each entry's `col` is its first byte within the row; its src_base is the
// source offset of the group's first row at that column (any byte
// alignment).
//
// Unit gather (kind | kUnitGather, in the unaligned row-gather section, for
// one receiver): lanes take 16-byte units of each segment's row rather than
// slots of the destination -- unit k of a segment of width w covers bytes
// [min(16k, w - 16), +16), so the last unit overlaps the one before it and
// rewrites the same bytes -- each one unaligned 16-byte load and one
// unaligned 16-byte store, with no shifts or merges.  A segment shorter
// than 16 bytes is one unit of w bytes, loaded from the aligned words that
// hold it and stored byte by byte; ds[0] = kUShortSegs marks such groups.  Fields: v0, v1 = units [v0, v1) of the region (unit v is unit
// v mod vpr of region row v / vpr); vpr = units per row with mul_vpr /
// sh_vpr; n1, n2 and their multipliers = the source levels; ss[0] = the
// region's first row in group numbering, ss[1] = the chunk's first region
// row; dst_base = that row's byte offset in the receivers' buffers; run =
// row bytes; batch / pad[2] = fast division by the nominal units per
// segment (a first guess); pad[0], pad[1] the segment entries, whose `pad`
// holds the segment's first unit within the row.
constexpr uint32_t kUnitGather = 0x08u;
constexpr uint32_t kUShortSegs = 1u;
struct Seg {
    uint64_t src_base;
    uint32_t ss[3];
    uint32_t buf;
    uint32_t col;  // unaligned gather: first byte of the segment within the row
    uint32_t pad;  // unit gather: first unit of the segment within the row
};
static_assert(sizeof(Seg) == 32, "segment entries are shared by host and device");
constexpr uint32_t kMaxSegs = 256;  // segment entries one gather chunk may stage

// Tile-transpose path (own section and kernel), for tasks whose source and
// destination layouts are contiguous along different tensor dimensions (a
// permuted local layout): A is the dimension contiguous in the sender's
// buffer, B the one contiguous in the receivers'.  A tile is kTileBytes /
// es elements along each of A and B: its rows (one per B index) are
// kTileBytes contiguous source bytes, its columns (one per A index)
// kTileBytes contiguous destination bytes.  A chunk is a range of tiles of a
// piece (tile t: tb = t mod ntb fastest, then ta, then the outer levels o1,
// o2).  Fields: kind = log2 es | kTAlignLoad | kTAlignStore | (log2 of the
// width factor along B) << 6; ss[0] = sender
// stride of B, ds[0] = receiver stride of A; ss[1], ds[1] and ss[2], ds[2]
// the outer levels o1 (inner) and o2; vpr = ntb, n1 = nta, n2 = extent of o1
// (with their fast divisions); run = extent of A, batch = extent of B
// (elements); v0, v1 the tiles; src_base/dst_base, src_rel0/dst_rel0 as
// usual, for tile v0's origin.  The aligned flags say that every tile row
// (column) starts on a 16-byte boundary, so whole 16-byte vectors of it are
// loaded (stored) at once; otherwise elements move one by one.
constexpr uint32_t kTileBytes = 128;
constexpr uint32_t kTAlignLoad = 0x10u;
constexpr uint32_t kTAlignStore = 0x20u;
constexpr uint32_t tile_elems(uint32_t es) { return kTileBytes / es; }
// A tile spans 1, 2 or 4 x kTileBytes along B (kind bits 6-7 hold log2 of
// that factor): wide enough to write whole destination rows of up to 512
// bytes, so each tile fills every cache line of the rows it writes.  Its
// LDS image is (B extent) rows of kTileBytes.
constexpr uint32_t tile_wide_log2(uint32_t kind) { return (kind >> 6) & 3u; }
constexpr uint32_t tile_rows(uint32_t es, uint32_t kind) { return tile_elems(es) << tile_wide_log2(kind); }

// Relative offsets (sender, receiver) of tile t's origin from the chunk's
// first tile (mod 2^32), and the tile's (ta, tb) indices.
struct TileAt {
    uint32_t src, dst, ta, tb;
};

constexpr TileAt tile_offsets(const Desc &d, uint32_t t, uint32_t es) {
    const uint32_t r = fastdiv(t, d.mul_vpr, d.sh_vpr);
    const uint32_t tb = t - r * d.vpr;
    const uint32_t o = fastdiv(r, d.mul_n1, d.sh_n1);
    const uint32_t ta = r - o * d.n1;
    const uint32_t o2 = fastdiv(o, d.mul_n2, d.sh_n2);
    const uint32_t o1 = o - o2 * d.n2;
    const uint32_t te = tile_elems(es), tr = tile_rows(es, d.kind);
    const uint32_t s = tb * tr * d.ss[0] + ta * kTileBytes + o1 * d.ss[1] + o2 * d.ss[2];
    const uint32_t u = ta * te * d.ds[0] + tb * (tr * es) + o1 * d.ds[1] + o2 * d.ds[2];
    return TileAt{s - d.src_rel0, u - d.dst_rel0, ta, tb};
}

// LDS byte offset of byte `o` of 16-byte column slot c in tile row r: rows
// are kTileBytes apart, and the slot is XOR-swizzled by the row's group of
// 16 / es rows, so the column reads of the store phase (16 / es rows of one
// slot per output vector) of a 128-byte-wide tile hit distinct banks.  In
// wider tiles 32 lanes read one column through 8 slots and conflict; a
// conflict-free lane order measured no faster (the kernel is not LDS-bound).
constexpr uint32_t tile_lds(uint32_t r, uint32_t c, uint32_t o, uint32_t es) {
    return r * kTileBytes + ((c ^ ((r / (16u / es)) & 7u)) << 4) + o;
}

// Outer-level indices of a row (level 1 = innermost outer level).
template <int LEVELS>
constexpr void row_indices(const Desc &d, uint32_t row, uint32_t &i1, uint32_t &i2, uint32_t &i3) {
    if (LEVELS == 1) {
        i1 = row;
        i2 = 0;
        i3 = 0;
    } else {
        const uint32_t r2 = fastdiv(row, d.mul_n1, d.sh_n1);
        i1 = row - r2 * d.n1;
        if (LEVELS == 2) {
            i2 = r2;
            i3 = 0;
        } else {
            i3 = fastdiv(r2, d.mul_n2, d.sh_n2);
            i2 = r2 - i3 * d.n2;
        }
    }
}

// Offsets (sender, receiver) of vector v relative to the chunk's first vector.
struct Rel {
    uint32_t src;
    uint32_t dst;
};

// Offsets of the start of row `row` of the piece relative to the chunk's
// first vector (mod 2^32).
template <int LEVELS>
constexpr Rel row_offsets(const Desc &d, uint32_t row) {
    uint32_t s = 0;
    uint32_t t = 0;
    if (LEVELS == 1) {
        s += row * d.ss[0];
        t += row * d.ds[0];
    } else {
        const uint32_t r2 = fastdiv(row, d.mul_n1, d.sh_n1);
        const uint32_t r1 = row - r2 * d.n1;
        s += r1 * d.ss[0];
        t += r1 * d.ds[0];
        if (LEVELS == 2) {
            s += r2 * d.ss[1];
            t += r2 * d.ds[1];
        } else {
            const uint32_t r3 = fastdiv(r2, d.mul_n2, d.sh_n2);
            const uint32_t q2 = r2 - r3 * d.n2;
            s += q2 * d.ss[1] + r3 * d.ss[2];
            t += q2 * d.ds[1] + r3 * d.ds[2];
        }
    }
    return Rel{s - d.src_rel0, t - d.dst_rel0};
}

template <int LEVELS>
constexpr Rel chunk_offsets(const Desc &d, uint32_t v, uint32_t vbytes) {
    const uint32_t row = fastdiv(v, d.mul_vpr, d.sh_vpr);
    const uint32_t col = v - row * d.vpr;
    const Rel r = row_offsets<LEVELS>(d, row);
    return Rel{r.src + col * vbytes, r.dst + col * vbytes};
}

// v_alignbyte semantics: bytes [sh, sh+4) of the 8-byte value hi:lo.
constexpr uint32_t align_byte(uint32_t hi, uint32_t lo, uint32_t sh) {
    return uint32_t(((uint64_t(hi) << 32) | lo) >> (8u * sh));
}

}  // namespace rs
