// Internal declarations shared by the host codec and the device launchers.
#pragma once
#include <cstdint>

#include "hufflm.h"

namespace hl {

// Section offsets of a container: off_seg_bits holds one byte per segment
// (its stored length over its group's base), off_grp_off the u32 start (in
// 16-byte units) and base of every group, then the end of the last stream.
struct Layout {
  uint64_t n, n_seg, n_grp, L, off_seg_bits, off_grp_off, off_stream;
  uint32_t GR, GC;
};

// A group's stored segment lengths span at most this many bits over its base.
constexpr uint32_t kSegLenSpan = 255;

// Group g = rb*(L/GC) + cb: rows r0 .. r0+G-1 and column segments
// c0 .. c0+GC-1; segment mu = j*G + i is (r0 + i, c0 + j); `first` is the
// group-order number of its first segment.
struct GroupGeom {
  uint64_t r0, c0, first;
  uint32_t G, GC;
};
GroupGeom group_geom(uint64_t rows, uint64_t L, uint32_t GR, uint64_t g);
bool grp_rows_ok(uint64_t cols, uint32_t S, uint32_t GR);
uint32_t default_grp_rows(uint64_t cols, uint32_t S);

struct Header {
  uint64_t rows, cols, n_seg, n_grp, off_seg_bits, off_grp_off, off_stream, off_raw, total_bytes;
  uint32_t seg_len, grp_rows, max_grp_units, format, lmax;
  hl_codebook cb;      // format 0 (zero otherwise)
  hl_codebook8 cb8;    // format 1 (zero otherwise)
  hl_codebook16 cb16;  // format 2 (zero otherwise)
};

// Bytes of the raw plane: one per weight, or one sign bit per weight (float16).
inline uint64_t raw_bytes(uint64_t n, uint32_t format) { return format == HL_FORMAT_FP16 ? n / 8 : n; }

bool shape_ok(uint64_t rows, uint64_t cols, uint32_t S);
Layout make_layout(uint64_t rows, uint64_t cols, uint32_t S, uint32_t GR, uint32_t format);
// Reads the header and, in the whole-exponent format, the code-length section
// (needs 384 bytes); false if the fixed fields are wrong or bytes too few.
bool parse_header(const uint8_t* b, size_t bytes, Header* out);
bool header_consistent(const Header& h, uint64_t blob_bytes);
bool field_code_valid(const hl_field_code& fc, uint32_t lmax);
bool code8_valid(const hl_codebook8& cb);
bool code16_valid(const hl_codebook16& cb);
// Canonical code values of n symbols with lengths <= 16 (RFC 1951 Sec. 3.2.2).
void canonical_codes(const uint8_t* len, int n, uint32_t* code);
uint32_t default_seg_len(uint64_t cols);
// Full structural check of a host copy; fills the header and the longest
// segment (in code bits).
hl_status validate_blob(const uint8_t* b, size_t bytes, Header* out, uint32_t* max_seg_bits);

}  // namespace hl
