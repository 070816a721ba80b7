// gfx950 kernels of the Huff-LLM bf16 codec: decode-table build, decode to
// bf16, fused decode-GEMV, the uncompressed bf16 GEMV comparator, and their
// C-ABI launchers.
//
// Decoding follows the decoder of Huff-LLM Sec. 3.2: a window of bits at the
// start pointer is matched against the codebook, the symbol is emitted and the
// pointer advances by the code length; the raw sign is passed through and the
// fields are concatenated back into the 16-bit weight. Here the "CAM" is an
// 8192-entry table in LDS indexed by a 13-bit window that yields both codes of
// a weight (exponent low and high nibble) at once; pairs longer than 13 bits
// fall back to a bit-serial canonical decode. Weights are decoded only where
// they are multiplied (Sec. 1, Sec. 3.2): the fused kernel never writes them.
//
// Work mapping (container tiling in include/hufflm.h): one wavefront decodes
// one group = G rows x GC column segments (G*GC <= 64), lane mu owning the
// segment of row r0 + mu % G and column segment c0 + mu / G. Each lane's part
// of the group stream goes into a column of the wave's LDS region (word j of
// lane lam at row j, column lam), so that window reads never share an LDS
// bank between lanes. The vector and decode kernels also stage the raw
// sign/mantissa plane ([t/8][lane] in 8-byte units) and the activation slice
// in LDS; the matrix-core kernels keep raw bytes and activations in
// registers, prefetched steps ahead, and the persistent kernel loads the next
// group's stream words into registers while it decodes the current group (in
// its decode form it also decodes large matrices to bf16).
#include <hip/hip_runtime.h>
#include <hipblaslt/hipblaslt.h>

#include <algorithm>
#include <type_traits>
#include <cstring>
#include <mutex>

#include "hl_internal.h"
#include "hufflm.h"

namespace hl {

constexpr int kLutBits = 13;
constexpr int kLutN = 1 << kLutBits;   // joint window table entries
constexpr int kAuxWords = 64;          // canonical tables for the long-code path
constexpr int kAuxField = 24;          // words per field in the aux table
constexpr uint32_t kEsc = 0x80000080u; // entry of a pair longer than the window
constexpr uint32_t kElKnown = 1u << 16; // ... whose el code fits: its length in bits 8..11, el in 12..15
constexpr int kMaxWaves = 16;
constexpr uint32_t kCol = 64;          // row stride of the stream columns, in words

static_assert(HL_LUT_BYTES >= (kLutN + kAuxWords) * 4, "table size");

// Joint table entry: bits 0..4 = code bits of the (el, eh) pair, bits 23..30 =
// the exponent byte eh<<4|el (its place in a float32), all other bits zero.
// A window whose pair is longer than 13 bits maps to kEsc (bits 7 and 31),
// plus kElKnown with el's code length and value when el's code alone fits.
// Bit 31 makes the entry negative: one test of the OR of a window's four
// entries finds any escape; as a shift the entry moves nothing (bits 0..5 are
// zero). Bit 7 keeps escape entries distinct from pair lengths (at most 13).
// Aux table, per field f (0 = eh, 1 = el) at word f*24: [0] = nsym |
// single<<8 | maxlen<<16; [l], l = 1..15: first_code<<16 | count<<8 | offset;
// [16..19]: symbols sorted by (length, symbol), one byte each.
struct Aux {
  uint32_t w[kAuxWords];
};

// One field's canonical tables in the aux format above, for an alphabet of
// `alpha` symbols (16 or 32: the symbol bytes fill words 16..19 or 16..23).
static void fill_aux_field(uint32_t* w, const uint8_t* len, int alpha, int nsym, int single) {
  uint32_t code[32];
  canonical_codes(len, alpha, code);
  int maxl = 0;
  for (int s = 0; s < alpha; ++s) maxl = std::max(maxl, (int)len[s]);
  if (nsym == 1) maxl = 0;
  w[0] = (uint32_t)nsym | ((uint32_t)single << 8) | ((uint32_t)maxl << 16);
  int k = 0;
  uint8_t sorted[32] = {0};
  for (int l = 1; l <= 15; ++l) {
    int first = -1, cnt = 0, off = k;
    for (int s = 0; s < alpha; ++s) {
      if (nsym > 1 && len[s] == l) {
        if (first < 0) first = (int)code[s];
        sorted[k++] = (uint8_t)s;
        ++cnt;
      }
    }
    w[l] = ((uint32_t)(first < 0 ? 0 : first) << 16) | ((uint32_t)cnt << 8) | (uint32_t)off;
  }
  for (int i = 0; i < alpha; ++i) w[16 + i / 4] |= (uint32_t)sorted[i] << (8 * (i % 4));
}

static Aux make_aux(const hl_codebook& cb) {
  Aux a;
  std::memset(&a, 0, sizeof(a));
  fill_aux_field(a.w, cb.eh.len, 16, cb.eh.nsym, cb.eh.single);
  fill_aux_field(a.w + kAuxField, cb.el.len, 16, cb.el.nsym, cb.el.single);
  return a;
}


// ------------------------------------------------------------------ device

// Joint table and aux tables, at a fixed LDS address in every kernel that decodes.
__shared__ __attribute__((aligned(16))) uint32_t s_tab[kLutN + kAuxWords];
extern __shared__ uint32_t s_dyn[];

// One field, bit-serial canonical decode from `bits` (LSB = next bit), using
// at most `avail` bits. Returns the symbol or -1 if no code of <= avail bits
// matches.
__device__ inline int field_from_bits(const uint32_t* aux, uint32_t bits, uint32_t avail,
                                      uint32_t* used) {
  const uint32_t meta = aux[0];
  if ((meta & 0xFF) == 1) { *used = 0; return (int)((meta >> 8) & 0xFF); }
  const uint32_t maxl = (meta >> 16) & 0xFF;
  uint32_t code = 0;
  for (uint32_t l = 1; l <= maxl && l <= avail; ++l) {
    code = (code << 1) | ((bits >> (l - 1)) & 1u);
    const uint32_t w = aux[l];
    const uint32_t d = code - (w >> 16);
    if (d < ((w >> 8) & 0xFF)) {
      const uint32_t k = (w & 0xFF) + d;
      *used = l;
      return (int)((aux[16 + (k >> 2)] >> (8 * (k & 3))) & 0xFF);
    }
  }
  return -1;
}

// Builds the joint table: entry v decodes the 13-bit window v (bit 0 first).
__global__ void __launch_bounds__(256) lut_kernel(uint32_t* lut, Aux aux) {
  for (int v = threadIdx.x; v < kLutN; v += blockDim.x) {
    uint32_t ua = 0, ub = 0;
    const int b = field_from_bits(aux.w + kAuxField, (uint32_t)v, kLutBits, &ub);  // el first
    const int a = b < 0 ? -1 : field_from_bits(aux.w, (uint32_t)v >> ub, kLutBits - ub, &ua);
    lut[v] = b < 0   ? kEsc
             : a < 0 ? kEsc | kElKnown | (ub << 8) | ((uint32_t)b << 12)
                     : ((ua + ub) | ((uint32_t)((a << 4) | b) << 23));
  }
  for (int i = threadIdx.x; i < kAuxWords; i += blockDim.x) lut[kLutN + i] = aux.w[i];
}

// Whole-exponent code in canonical form: per length l = 1..13 the first code
// value, the number of codes and the index of the first of them in `sym`,
// the exponent values sorted by (length, value).
struct Aux8 {
  uint32_t nsym, single;
  uint32_t first[kLutBits + 1], count[kLutBits + 1], off[kLutBits + 1];
  uint8_t sym[256];
};

static Aux8 make_aux8(const hl_codebook8& cb) {
  Aux8 a;
  std::memset(&a, 0, sizeof(a));
  a.nsym = cb.nsym;
  a.single = cb.single;
  if (cb.nsym == 1) return a;
  uint32_t code[256];
  canonical_codes(cb.len, 256, code);
  uint32_t k = 0;
  for (int l = 1; l <= kLutBits; ++l) {
    a.off[l] = k;
    for (int s = 0; s < 256; ++s) {
      if (cb.len[s] != l) continue;
      if (a.count[l] == 0) a.first[l] = code[s];
      ++a.count[l];
      a.sym[k++] = (uint8_t)s;
    }
  }
  return a;
}

// Decode table of the whole-exponent format: entry v = the code that the
// 13-bit window v (bit 0 first) starts with, as its length in bits 0..4 and
// the exponent byte in bits 23..30, the entry format of the split table. A
// complete code of at most 13 bits matches every window; kEsc is left only
// for a damaged code. The aux words are zero (no long codes).
__global__ void __launch_bounds__(256) lut8_kernel(uint32_t* lut, Aux8 a) {
  for (int v = threadIdx.x; v < kLutN; v += blockDim.x) {
    uint32_t ent = kEsc;
    if (a.nsym == 1) {
      ent = a.single << 23;
    } else {
      uint32_t code = 0;
      for (uint32_t l = 1; l <= (uint32_t)kLutBits; ++l) {
        code = (code << 1) | (((uint32_t)v >> (l - 1)) & 1u);
        const uint32_t d = code - a.first[l];
        if (d < a.count[l]) {
          ent = l | ((uint32_t)a.sym[a.off[l] + d] << 23);
          break;
        }
      }
    }
    lut[v] = ent;
  }
  for (int i = threadIdx.x; i < kAuxWords; i += blockDim.x) lut[kLutN + i] = 0;
}

// Copies the joint table and the aux tables into LDS, four 16-byte loads in
// flight per thread.
__device__ inline void load_tables(const uint32_t* lut) {
  constexpr uint32_t kVec = (kLutN + kAuxWords) / 4;  // uint4 count
  const uint4* src = reinterpret_cast<const uint4*>(lut);
  uint4* dst = reinterpret_cast<uint4*>(s_tab);
  const uint32_t n = blockDim.x;
  for (uint32_t k = threadIdx.x; k < kVec; k += 4 * n) {
    const uint4 v0 = src[k];
    const uint4 v1 = k + n < kVec ? src[k + n] : v0;
    const uint4 v2 = k + 2 * n < kVec ? src[k + 2 * n] : v0;
    const uint4 v3 = k + 3 * n < kVec ? src[k + 3 * n] : v0;
    dst[k] = v0;
    if (k + n < kVec) dst[k + n] = v1;
    if (k + 2 * n < kVec) dst[k + 2 * n] = v2;
    if (k + 3 * n < kVec) dst[k + 3 * n] = v3;
  }
}

// The same copy as direct global-to-LDS transfers (16 bytes per lane, no
// registers): the caller waits for them (vmcnt) before its barrier.
constexpr uint32_t kTabVec = (kLutN + kAuxWords) / 4;  // 16-byte pieces

// Block barrier for LDS data only: waits for this wave's LDS accesses, not for
// its outstanding global loads and copies (gfx950 barriers do not need them).
__device__ inline void block_sync_lds() {
  __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4));  // lgkmcnt(0)
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

__device__ inline void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}
// s_waitcnt through the builtin, so that the compiler's own wait insertion
// knows what has completed. gfx9 encoding: vmcnt in bits 3..0 and 15..14,
// expcnt in 6..4, lgkmcnt in 11..8; a field at its maximum does not wait.
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
constexpr int kWaitLgkm0 = 15 | (3 << 14) | (7 << 4);
__device__ inline void wait_vm0() {
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  asm volatile("" ::: "memory");
}
__device__ inline void wait_vm1() {
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(1));
  asm volatile("" ::: "memory");
}
__device__ inline void wait_lgkm0() {
  __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
  asm volatile("" ::: "memory");
}

// Direct global-to-LDS copies (no VGPR staging): every lane moves `size`
// bytes from its own address to lds_base + lane * size; lds_base is
// wave-uniform.
__device__ inline void dma16(const void* src, uint32_t* lds_base) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)lds_base, 16, 0, 0);
}
__device__ inline void dma4(const void* src, uint32_t* lds_base) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)lds_base, 4, 0, 0);
}

__device__ inline void table_dma(const uint32_t* lut) {
  const uint32_t n = blockDim.x, w0 = threadIdx.x & ~63u, lane = threadIdx.x & 63;
  for (uint32_t k0 = w0; k0 < kTabVec; k0 += n)
    if (k0 + lane < kTabVec) dma16(lut + (k0 + lane) * 4, s_tab + k0 * 4);
}

// ---- stream columns
// A lane's column pointer `sc` addresses its row-0 word; word j is sc[j*64].
// Row 0 is padding: a lane's first stream word sits in row 1, so positions
// start at 32 + (start bit within that word).
//
// Positions: pos2 = column bit position minus 2, so that the window's low
// 15 bits hold two old bits and the 13-bit peek already scaled by 4, the
// byte offset of a table entry. In the fast loop pos2 accumulates whole table
// entries; only bits 0..22 are the position (exponent bytes pile up above bit
// 22), so positions are read through kPosMask.
constexpr uint32_t kPosMask = 0x7FFFFFu;

__device__ inline uint32_t col_word(const uint32_t* sc, uint32_t j) { return sc[j * kCol]; }

// Bit-serial decode of one field from the lane's column at bit p (advanced);
// rows beyond jmax are read as row jmax.
__device__ inline uint32_t slow_field(const uint32_t* sc, const uint32_t* aux, uint32_t& p, uint32_t jmax) {
  const uint32_t meta = aux[0];
  if ((meta & 0xFF) == 1) return (meta >> 8) & 0xFF;
  const uint32_t maxl = (meta >> 16) & 0xFF;
  uint32_t code = 0;
  for (uint32_t l = 1; l <= maxl; ++l) {
    code = (code << 1) | ((col_word(sc, min(p >> 5, jmax)) >> (p & 31)) & 1u);
    ++p;
    const uint32_t w = aux[l];
    const uint32_t d = code - (w >> 16);
    if (d < ((w >> 8) & 0xFF)) {
      const uint32_t k = (w & 0xFF) + d;
      return (aux[16 + (k >> 2)] >> (8 * (k & 3))) & 0xFF;
    }
  }
  return 0;  // no code matched: damaged stream, decode continues safely
}

// 64-bit window of column bits [pos2, pos2 + 64); jmax bounds the first row
// read (two more rows follow) so that a damaged stream cannot leave the region.
__device__ inline uint64_t load_window(const uint32_t* sc, uint32_t pos2, uint32_t jmax) {
  const uint32_t j = min((pos2 & kPosMask) >> 5, jmax);
  const uint32_t a = col_word(sc, j), b = col_word(sc, j + 1), c = col_word(sc, j + 2);
  return ((uint64_t)__builtin_amdgcn_alignbit(c, b, pos2) << 32) | __builtin_amdgcn_alignbit(b, a, pos2);
}

__device__ inline uint32_t lut_at(uint32_t w) {
  return *reinterpret_cast<const uint32_t*>(reinterpret_cast<const uint8_t*>(s_tab) +
                                            (w & ((kLutN - 1) << 2)));
}

// Window shift by a table entry: bits 0..5 of the entry are the pair length
// (0 for an escape); v_lshrrev_b64 reads only those bits of its count.
__device__ inline uint64_t shift_window(uint64_t w, uint32_t ent) { return w >> (ent & 63u); }

// Careful path for the four weights of a window: the pairs one after
// another, each pair longer than the table's 13 bits decoded field by field
// from the window's bits (el from the table entry when its code fits in 13
// bits, else bit by bit, then eh bit by bit). The window is read again at the
// pair's position when fewer than 13 of its 62 bits are left (fewer than 30
// for a long pair). A rolled loop keeps the (cold, inlined) code small.
// pos2: the window's clean start position (no exponent bits above bit 22).
__device__ __attribute__((always_inline)) inline void careful4(uint32_t sc_off, uint32_t jmax, uint32_t pos2,
                                                              uint32_t* e) {
  asm volatile("" ::: "memory");  // keeps its table reads inside the (cold) path
  const uint32_t* sc = s_dyn + sc_off;
  const uint32_t* aux = s_tab + kLutN;
  uint32_t r[4] = {0, 0, 0, 0};
  uint64_t W = 0;
  uint32_t used = 64;  // bits of W consumed (none loaded yet)
#pragma unroll 1
  for (uint32_t k = 0; k < 4; ++k) {
    if (used > 62 - 13) {
      W = load_window(sc, pos2, jmax);
      used = 0;
    }
    uint32_t ent = lut_at((uint32_t)W);
    if (ent & kEsc) {
      if (used > 62 - 30) {
        W = load_window(sc, pos2, jmax);
        used = 0;
      }
      const uint32_t bits = (uint32_t)(W >> 2);  // the code bits from the position on
      uint32_t ub = 0, ua = 0;
      int b;
      if (ent & kElKnown) {  // the table decoded el: only eh is left, a code of a few bits
        ub = (ent >> 8) & 0xF;
        b = (int)((ent >> 12) & 0xF);
      } else {
        b = field_from_bits(aux + kAuxField, bits, 32, &ub);  // el first
      }
      int a = b < 0 ? -1 : field_from_bits(aux, bits >> ub, 32 - ub, &ua);
      if (b < 0) b = 0, ub = 0;  // no code matches (a damaged stream): decode on, in bounds
      if (a < 0) a = 0, ua = 0;
      ent = (ua + ub) | ((uint32_t)((a << 4) | b) << 23);
    }
    W = shift_window(W, ent);
    used += ent & 0xFF;
    pos2 += ent & 0xFF;
#pragma unroll
    for (int j = 0; j < 4; ++j) r[j] = k == (uint32_t)j ? ent : r[j];
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) e[j] = r[j];
}

// A pair longer than the table window, within the fast path: el from the
// escape entry, eh bit by bit from the window. Left as an escape (for the
// careful path) when el's code is longer than the table window, when no eh
// code matches, or when the pair runs past the window's 62 bits (`used` of
// them are consumed).
__device__ __attribute__((always_inline)) inline uint32_t long_pair(uint32_t ent, uint64_t W, uint32_t used) {
  if (!(ent & kElKnown)) return ent;
  const uint32_t ub = (ent >> 8) & 0xF, b = (ent >> 12) & 0xF;
  uint32_t ua = 0;
  const int a = field_from_bits(s_tab + kLutN, (uint32_t)(W >> 2) >> ub, 32 - ub, &ua);
  if (a < 0 || used + ub + ua > 62) return ent;
  return (ua + ub) | ((uint32_t)((a << 4) | b) << 23);
}

// The four table reads of the window W0 again, resolving long pairs.
__device__ __attribute__((always_inline)) inline void redo4(uint64_t W0, uint32_t* e) {
  uint64_t W = W0;
  uint32_t used = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    uint32_t ent = lut_at((uint32_t)W);
    if ((int)ent < 0) ent = long_pair(ent, W, used);
    W = shift_window(W, ent);
    used += ent & 0x3F;
    e[k] = ent;
  }
}

// Four table reads from the 64-bit window W (four pairs of at most 13 bits
// fit): table entries e[4] (bits 23..30 = exponent byte), p advanced by the
// whole entries. Bits 0..22 of a position are the bit position; the exponent
// bytes pile up above them and are never read. An escape entry (a pair longer
// than the table window) has bit 31 set and advances nothing useful; the
// caller tests for it.
__device__ inline void lookup4(uint64_t W, uint32_t& p, uint32_t* e) {
  e[0] = lut_at((uint32_t)W);
  W = shift_window(W, e[0]);
  e[1] = lut_at((uint32_t)W);
  W = shift_window(W, e[1]);
  e[2] = lut_at((uint32_t)W);
  W = shift_window(W, e[2]);
  e[3] = lut_at((uint32_t)W);
  p = p + e[0] + e[1] + e[2] + e[3];
}

// The four weights of window W (at clean position p) again, resolving long
// pairs (from the window's bits, else by the careful path); p advanced.
__device__ __attribute__((always_inline)) inline void resolve4(uint64_t W, uint32_t sc_off, uint32_t jmax,
                                                              uint32_t& p, uint32_t* e) {
  redo4(W, e);
  if ((int)(e[0] | e[1] | e[2] | e[3]) < 0) careful4(sc_off, jmax, p, e);
  p = (p + e[0] + e[1] + e[2] + e[3]) & kPosMask;
}

// 64 bits of the three words (c, b, a) from bit p % 32 of a on.
__device__ inline uint64_t funnel64(uint32_t c, uint32_t b, uint32_t a, uint32_t p) {
  return ((uint64_t)__builtin_amdgcn_alignbit(c, b, p) << 32) | __builtin_amdgcn_alignbit(b, a, p);
}

// Decodes 8 weights: four words of the lane's column are read at once; the
// first window is bits [p, p + 64) of them, the second starts where the first
// four pairs ended, within the same four words when that is at most one word
// further (a rare longer advance reads its window from the column). jmax - 1
// bounds the first of the four rows (columns hold three rows of overrun).
// One wave-uniform test of the OR of the eight entries finds any escape; a
// lane that had one decodes the window with the escape again from its
// registers (and, after an escape in the first, the second window from the
// corrected position).
__device__ inline void decode8(const uint32_t* sc, uint32_t sc_off, uint32_t jmax, uint32_t& pos2, uint32_t* e) {
  uint32_t p = pos2;
  const uint32_t j = min((p & kPosMask) >> 5, jmax - 1);
  const uint32_t w0 = col_word(sc, j), w1 = col_word(sc, j + 1), w2 = col_word(sc, j + 2), w3 = col_word(sc, j + 3);
  lookup4(funnel64(w2, w1, w0, p), p, e);
  const uint32_t pm = p;  // after the first four
  const uint32_t rel = ((p & kPosMask) >> 5) - j;  // rows the position moved (wraps if it went back)
  const bool r1 = rel != 0;  // selects, not a branch
  uint64_t W = funnel64(r1 ? w3 : w2, r1 ? w2 : w1, r1 ? w1 : w0, p);
  if (__builtin_expect(__builtin_amdgcn_ballot_w64(rel > 1) != 0, 0))
    if (rel > 1) W = load_window(sc, p, jmax);
  lookup4(W, p, e + 4);
  const uint32_t any = e[0] | e[1] | e[2] | e[3] | e[4] | e[5] | e[6] | e[7];
  if (__builtin_expect(__builtin_amdgcn_ballot_w64((int)any < 0) != 0, 0)) {
    if ((int)any < 0) {
      if ((int)(e[0] | e[1] | e[2] | e[3]) < 0) {
        p = pos2 & kPosMask;
        resolve4(funnel64(w2, w1, w0, p), sc_off, jmax, p, e);
        W = load_window(sc, p, jmax);
      } else {
        p = pm & kPosMask;
      }
      resolve4(W, sc_off, jmax, p, e + 4);
    }
  }
  pos2 = p;
}

// ---- bounded pairs: every weight's codes fit 11 bits
// When the longest code pair of a matrix is at most kBpBits bits, an
// 11-bit window holds a whole pair: the table has 2048 entries (the joint
// table's first 2048, whose upper window bits are zero) and is kept in LDS
// in kBpCopies copies, entry v of copy c at word v*kBpCopies + c, lane l
// reading copy l % kBpCopies: the 32 lanes of a half-wave then spread over
// the banks by copy as well as by entry, instead of colliding on the banks
// of the short, frequent pairs. Four pairs then move the position at most 44
// bits, so the four column words of a step always hold the second window
// (no long-move branch), and no entry is an escape (no escape test).
// Positions here are column bit positions minus 5: the window's low 16 bits
// then hold five old bits and the 11-bit index already scaled by 32, the
// byte offset of the entry's first copy.
#ifndef HL_BP_BITS
#define HL_BP_BITS HL_PAIR_MAX
#endif
constexpr int kBpBits = HL_BP_BITS;
static_assert(kBpBits <= (int)HL_PAIR_MAX && kBpBits >= 9, "table window");
constexpr uint32_t kBpN = 1u << kBpBits;
constexpr uint32_t kBpCopies = 1u << (14 - kBpBits);
constexpr uint32_t kBpShift = 16 - kBpBits;  // log2 of an entry's bytes over all copies
constexpr uint32_t kBpWords = kBpN * kBpCopies;  // 64 KB

// The replicated table, a static LDS array of its own: at a fixed address
// in the kernels that use it (no other static LDS there), so that a lookup's
// address is one and-or of the window and the lane's copy offset.
__shared__ __attribute__((aligned(32))) uint32_t s_bp[kBpWords];

// The replicated table is filled from the global joint table (its first
// kBpN entries) in two halves: the thread's entries are loaded into registers
// (blocks of at least kBpMinThreads threads: at most kBpPerThread each) at the
// kernel's start, and stored to LDS, in kBpCopies copies, once other loads
// have been requested behind them.
constexpr uint32_t kBpMinThreads = 512;
constexpr uint32_t kBpPerThread = kBpN / kBpMinThreads;

__device__ inline void bp_table_load(const uint32_t* lut, uint32_t (&te)[kBpPerThread]) {
#pragma unroll
  for (uint32_t k = 0; k < kBpPerThread; ++k) {
    const uint32_t v = threadIdx.x + k * blockDim.x;
    te[k] = v < kBpN ? lut[v] : 0u;
  }
}

__device__ inline void bp_table_store(const uint32_t (&te)[kBpPerThread]) {
#pragma unroll
  for (uint32_t k = 0; k < kBpPerThread; ++k) {
    const uint32_t v = threadIdx.x + k * blockDim.x, e = te[k];
    if (v < kBpN) {
      uint4* d = reinterpret_cast<uint4*>(s_bp + v * kBpCopies);
#pragma unroll
      for (uint32_t c = 0; c < kBpCopies / 4; ++c) d[c] = make_uint4(e, e, e, e);
    }
  }
}

__device__ inline uint32_t bp_at(uint32_t w, uint32_t lane_off) {
  const uint32_t off = (w & ((kBpN - 1) << kBpShift)) | lane_off;
  return *reinterpret_cast<const uint32_t*>(reinterpret_cast<const uint8_t*>(s_bp) + off);
}

// Four table reads from the window W, shifted past each pair read (W ends
// shifted past all four).
__device__ inline void bp_lookup4(uint64_t& W, uint32_t* e, uint32_t lane_off) {
  e[0] = bp_at((uint32_t)W, lane_off);
  W = shift_window(W, e[0]);
  e[1] = bp_at((uint32_t)W, lane_off);
  W = shift_window(W, e[1]);
  e[2] = bp_at((uint32_t)W, lane_off);
  W = shift_window(W, e[2]);
  e[3] = bp_at((uint32_t)W, lane_off);
}

// decode8 for bounded pairs: no branch. The first window is bits [p, p + 64)
// of four column words; the four pairs read from it take at most 44 bits,
// and the second window is what is left of it with the next 32 bits of the
// words (bits [p + 64, p + 96)) put right behind: at least 52 bits, more than
// the 49 its four lookups can reach. (Fields of one symbol have 0-bit codes:
// four pairs take at least 4 bits, except where both fields have one symbol,
// and then every window reads one and the same entry, so the refill's place
// does not matter.) jmax - 1
// bounds the first of the four rows read (columns hold three rows of overrun).
__device__ inline void bp_decode8(const uint32_t* sc, uint32_t jmax, uint32_t& pos5, uint32_t* e,
                                  uint32_t lane_off) {
  const uint32_t p = pos5;
  const uint32_t j = min((p & kPosMask) >> 5, jmax - 1);
  const uint32_t w0 = col_word(sc, j), w1 = col_word(sc, j + 1), w2 = col_word(sc, j + 2), w3 = col_word(sc, j + 3);
  uint64_t W = funnel64(w2, w1, w0, p);
  const uint32_t t = __builtin_amdgcn_alignbit(w3, w2, p);
  bp_lookup4(W, e, lane_off);
  W = shift_window(W, e[3]);
  const uint32_t p4 = p + e[0] + e[1] + e[2] + e[3];
  W |= (uint64_t)t << ((p - p4) & 63u);  // 64 - (bits of the four pairs)
  bp_lookup4(W, e + 4, lane_off);
  pos5 = p4 + e[4] + e[5] + e[6] + e[7];
}

// Packed bf16 pair (weights k, k+1 of a raw dword) from two table entries.
__device__ inline uint32_t pack_pair(uint32_t rawdw, int k, uint32_t e0, uint32_t e1) {
  const uint32_t b0 = (uint32_t)(k & 3), b1 = (uint32_t)((k + 1) & 3);
  const uint32_t P = __builtin_amdgcn_perm(rawdw, rawdw, b0 | (b0 << 8) | (b1 << 16) | (b1 << 24));
  const uint32_t E = __builtin_amdgcn_perm(e1, e0, 0x07060302u);
  return (P & 0x807F807Fu) | (E & 0x7F807F80u);
}

// float32 weight k of a raw dword from its table entry.
__device__ inline float weight_f32(uint32_t rawdw, int k, uint32_t e) {
  const uint32_t b = (uint32_t)(k & 3);
  const uint32_t M = __builtin_amdgcn_perm(rawdw, rawdw, 0x00000C0Cu | (b << 16) | (b << 24));
  return __uint_as_float((M & 0x807FFFFFu) | (e & 0x7F800000u));
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ inline float dot2(uint32_t w, uint32_t x, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w),
                                         __builtin_bit_cast(bf16x2_t, x), acc, false);
}

// Wait states after a matrix instruction before the next instruction may
// overwrite its A or B operand registers. Measured on gfx950: with the
// packed weights of the next step written into the A operand's registers by
// the instruction right after v_mfma_f32_16x16x32_bf16, the product
// intermittently used the new values (whole row blocks wrong); the compiler
// placed no wait states there. Five are enough and cost nothing measurable
// (the other waves of the SIMD issue meanwhile).
__device__ inline void mfma_operand_guard() { asm volatile("s_nop 4"); }

// ------------------------------------------------------------------ staging

struct GroupArgs {
  const uint8_t* seg_len8;   // per segment: its stored length over its group's base
  const uint32_t* grp_meta;  // per group: stream start (16-byte units), base; then the end
  const uint4* stream;
  const uint8_t* raw;
  const uint32_t* lut;   // global copy: kLutN entries + aux
  uint32_t rows, cols, S, L, GR, GC, CB, RB, stream_units, max_units;
  uint32_t col_rows;     // rows of the stream columns (row 0 = padding)
  // float16 format: LDS layout of its decode tables (see Tab16)
  uint32_t t16_mask[3];  // window index mask of the ml, e, mh tables (bytes)
  uint32_t t16_base[3];  // their byte offsets
  uint32_t t16_aux;      // word offset of the bit-serial tables
  uint32_t t16_words;    // words of all tables (a multiple of 4)
};

// Group geometry and its metadata (segment length of the lane, stream units).
struct Meta {
  uint64_t first;  // group-order number of the group's first segment
  uint32_t r0, G, N, c0;
  uint32_t nbw;    // the dword holding the lane's one-byte segment length
  uint32_t u0, units;
};

// Which word of a group's table entry a lane loads: lane 0 the group's
// stream start, lane 1 its end (the next group's start), lane 2 its base.
__device__ inline uint32_t meta_pick(uint32_t lane) { return lane == 1 ? 2u : lane == 2 ? 1u : 0u; }

// Group g's geometry, and its metadata loads (vector loads, counted by vmcnt).
__device__ inline Meta load_meta(const GroupArgs& a, uint32_t g, uint32_t lane) {
  Meta m;
  const uint32_t rb = g / a.CB;
  m.c0 = (g - rb * a.CB) * a.GC;
  m.r0 = rb * a.GR;
  m.G = min(a.GR, a.rows - m.r0);
  m.N = m.G * a.GC;
  m.first = (uint64_t)m.r0 * a.L + (uint64_t)m.c0 * m.G;
  // A whole dword, used as loaded (no conversion that would wait on it here);
  // the byte is picked and masked to lanes < N at use. The dword of the last
  // segments reaches at most 3 bytes past the lengths table, into the
  // padding before the group table (the lengths end off a 4-byte boundary
  // only where the next section's 64-byte alignment leaves padding).
  m.nbw = reinterpret_cast<const uint32_t*>(a.seg_len8)[(m.first + min(lane, m.N - 1)) >> 2];
  m.u0 = a.grp_meta[2 * g + meta_pick(lane)];
  m.units = 0;
  return m;
}

__device__ inline uint32_t wave_max(uint32_t v) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, d, 64));
  return v;
}

// Copies the group's stream into the lane columns of region `cols`; returns
// the lane's pos2 (column bit position - 2).
// Group start and length (lanes 0 and 1 of the metadata, made wave-uniform so
// that copies address as scalar base + 32-bit lane offset), and the lane's
// first stream word ws and bit bit0 (segment lengths prefix-summed in lane
// order); returns the lane's code bits.
__device__ inline uint32_t stream_start(const GroupArgs& a, Meta& m, uint32_t lane, uint32_t& ws,
                                        uint32_t& bit0) {
  uint32_t v0 = (uint32_t)__builtin_amdgcn_readlane((int)m.u0, 0);
  uint32_t v1 = (uint32_t)__builtin_amdgcn_readlane((int)m.u0, 1);
  const uint32_t base = (uint32_t)__builtin_amdgcn_readlane((int)m.u0, 2);
  v0 = min(v0, a.stream_units);
  v1 = min(max(v1, v0), a.stream_units);
  m.u0 = v0;
  m.units = min(v1 - v0, a.max_units);
  const uint32_t byte = (uint32_t)(m.first + min(lane, m.N - 1)) & 3u;
  const uint32_t nb = lane < m.N ? base + ((m.nbw >> (8 * byte)) & 0xFFu) : 0u;
  uint32_t incl = nb;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t t = __shfl_up(incl, d, 64);
    if ((int)lane >= d) incl += t;
  }
  const uint32_t start = min(incl - nb, m.units * 128u);
  ws = start >> 5;
  bit0 = start & 31;
  return nb;
}

// Copies the group's stream into the lane columns of region `cols` (as many
// rows as the longest lane needs); returns the lane's pos2 (column bit
// position - 2).
__device__ inline uint32_t issue_stream(const GroupArgs& a, uint32_t* cols, Meta& m, uint32_t lane) {
  uint32_t ws, bit0;
  const uint32_t nb = stream_start(a, m, lane, ws, bit0);
  // words the lane's windows read: its bits plus two words of window overrun
  const uint32_t nw = ((bit0 + nb + 31) >> 5) + 2;
  const uint32_t J = m.units ? min(wave_max(nw), a.col_rows - 1) : 0u;
  const uint8_t* src = reinterpret_cast<const uint8_t*>(a.stream + m.u0);  // uniform
  const uint32_t last = m.units * 4 - 1;
  // 32-bit byte offsets, so that the copy addresses as scalar base + lane offset
  for (uint32_t j = 0; j < J; ++j) dma4(src + (uint32_t)(min(ws + j, last) * 4u), cols + (j + 1) * kCol);
  return 30u + bit0;
}

typedef uint32_t u32x4_a4 __attribute__((ext_vector_type(4), aligned(4)));

// The group's stream words for the lane columns, loaded into registers: JT
// words per lane from its first word on (four per load). Words past the
// group's stream are read from what follows it in the container (the next
// group's stream or the raw plane, at most JT words on), as window overrun
// only; a group without stream bits reads its raw bytes. Returns the lane's
// pos2.
template <int JT>
__device__ inline uint32_t stream_load(const GroupArgs& a, Meta& m, uint32_t lane, u32x4_a4 (&sw)[JT / 4]) {
  uint32_t ws, bit0;
  stream_start(a, m, lane, ws, bit0);
  const uint32_t* base = m.units ? reinterpret_cast<const uint32_t*>(a.stream + m.u0)
                                 : reinterpret_cast<const uint32_t*>(a.raw + m.first * a.S);
  const uint32_t w0 = m.units ? ws : 0u;
#pragma unroll
  for (int k = 0; k < JT / 4; ++k) sw[k] = *reinterpret_cast<const u32x4_a4*>(base + w0 + 4 * k);
  return 30u + bit0;
}

// Writes the words of stream_load to the lane's column (rows 1..JT).
template <int JT>
__device__ inline void stream_store(uint32_t* cols, const u32x4_a4 (&sw)[JT / 4], uint32_t lane) {
#pragma unroll
  for (int k = 0; k < JT / 4; ++k) {
    cols[(4 * k + 1) * kCol + lane] = sw[k].x;
    cols[(4 * k + 2) * kCol + lane] = sw[k].y;
    cols[(4 * k + 3) * kCol + lane] = sw[k].z;
    cols[(4 * k + 4) * kCol + lane] = sw[k].w;
  }
}

// Copies the group's raw plane (N*S bytes) into `raw_lds`.
__device__ inline void issue_raw(const GroupArgs& a, uint32_t* raw_lds, const Meta& m, uint32_t lane) {
  const uint32_t bytes = m.N * a.S;
  const uint8_t* src = a.raw + m.first * a.S;
  if ((a.S & 15) == 0) {
    const uint32_t n = bytes / 16;
    for (uint32_t k0 = 0; k0 < n; k0 += 64)
      if (k0 + lane < n) dma16(src + (uint64_t)(k0 + lane) * 16, raw_lds + k0 * 4);
  } else {
    const uint32_t n = bytes / 4;
    for (uint32_t k0 = 0; k0 < n; k0 += 64)
      if (k0 + lane < n) dma4(src + (uint64_t)(k0 + lane) * 4, raw_lds + k0);
  }
}

// ------------------------------------------------------------------ decode

// Decode to bf16. Waves take groups in turn; region per wave: stream columns
// then the raw plane.
__global__ void __launch_bounds__(1024) decode_kernel(GroupArgs a, uint16_t* out) {
  const uint32_t lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t waves = blockDim.x >> 6;
  const uint32_t per_wave = a.col_rows * kCol + 16 * a.S;
  uint32_t* cols = s_dyn + wave * per_wave;
  uint32_t* raw_lds = cols + a.col_rows * kCol;
  const uint32_t sc_off = wave * per_wave + lane;
  const uint32_t* sc = s_dyn + sc_off;
  const uint32_t jmax = a.col_rows - 3;
  const uint32_t n_grp = a.RB * a.CB;
  const uint32_t stride = gridDim.x * waves;
  uint32_t g = blockIdx.x * waves + wave;
  Meta m;
  if (g < n_grp) m = load_meta(a, g, lane);
  load_tables(a.lut);
  __syncthreads();
  for (; g < n_grp; g += stride) {
    uint32_t pos2 = issue_stream(a, cols, m, lane);
    issue_raw(a, raw_lds, m, lane);
    const Meta cur = m;
    if (g + stride < n_grp) {
      m = load_meta(a, g + stride, lane);
      wait_vm1();
    } else {
      wait_vm0();
    }
    wave_sync_lds();
    if (lane < cur.N) {
      const uint2* rl = reinterpret_cast<const uint2*>(raw_lds) + lane;
      const uint32_t i = lane % cur.G, j = lane / cur.G;
      uint16_t* o = out + (uint64_t)(cur.r0 + i) * a.cols + (uint64_t)(cur.c0 + j) * a.S;
      for (uint32_t t = 0; t < a.S; t += 8) {
        const uint2 rw = rl[(t >> 3) * cur.N];
        uint32_t e[8];
        decode8(sc, sc_off, jmax, pos2, e);
        uint4 v;
        v.x = pack_pair(rw.x, 0, e[0], e[1]);
        v.y = pack_pair(rw.x, 2, e[2], e[3]);
        v.z = pack_pair(rw.y, 0, e[4], e[5]);
        v.w = pack_pair(rw.y, 2, e[6], e[7]);
        *reinterpret_cast<uint4*>(o + t) = v;
      }
    }
    wait_lgkm0();
    wave_sync_lds();
  }
}

// ------------------------------------------------------------------ fused GEMV

struct GemvArgs {
  GroupArgs g;
  const void* x;
  float* y;
  float* partial;     // workspace: KS x B x (RB*64) partial sums (KS > 1)
  uint32_t* counter;  // workspace: RB arrival counters, zero between calls
  uint32_t C;         // column blocks per block
  uint32_t KS;        // blocks per row block
  uint32_t x_words;   // LDS words of one wave's activation slice
  uint32_t B;         // batch rows
};

// Copies x[b][c0*S .. (c0+GC)*S) for every batch row into xs ([batch][GC*S]).
template <int B, bool XBF16>
__device__ inline void issue_x(const GemvArgs& p, uint32_t* xs, uint32_t c0, uint32_t lane) {
  constexpr uint32_t kXPer = XBF16 ? 8 : 4;  // activations per 16 bytes
  const uint32_t per_row = p.g.GC * p.g.S / kXPer, total = per_row * B;
  const uint4* xsrc = reinterpret_cast<const uint4*>(p.x);
  const uint32_t row_u4 = p.g.cols / kXPer, c0_u4 = c0 * p.g.S / kXPer;
  for (uint32_t k0 = 0; k0 < total; k0 += 64) {
    const uint32_t k = k0 + lane;
    if (k < total) {
      const uint32_t b = k / per_row, j = k - b * per_row;
      dma16(xsrc + (uint64_t)b * row_u4 + c0_u4 + j, xs + k0 * 4);
    }
  }
}

// Multiply-accumulate of 8 decoded weights (entries e, raw dword pair rw)
// with the activations x[b][t .. t+8) of the lane's slice; xs points at the
// lane's segment in batch row 0, ldx is the slice's row length.
template <int B, bool XBF16>
__device__ inline void mac8(float* acc, const uint32_t* e, uint2 rw, const uint32_t* xs, uint32_t ldx,
                            uint32_t t) {
  if constexpr (XBF16) {
    const uint32_t w0 = pack_pair(rw.x, 0, e[0], e[1]);
    const uint32_t w1 = pack_pair(rw.x, 2, e[2], e[3]);
    const uint32_t w2 = pack_pair(rw.y, 0, e[4], e[5]);
    const uint32_t w3 = pack_pair(rw.y, 2, e[6], e[7]);
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const uint4 xv = *reinterpret_cast<const uint4*>(xs + b * (ldx / 2) + t / 2);
      float s = acc[b];
      s = dot2(w0, xv.x, s);
      s = dot2(w1, xv.y, s);
      s = dot2(w2, xv.z, s);
      s = dot2(w3, xv.w, s);
      acc[b] = s;
    }
  } else {
    float wf[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) wf[k] = weight_f32(k < 4 ? rw.x : rw.y, k, e[k]);
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const float* xf = reinterpret_cast<const float*>(xs) + b * ldx + t;
      const float4 x0 = *reinterpret_cast<const float4*>(xf);
      const float4 x1 = *reinterpret_cast<const float4*>(xf + 4);
      float s = acc[b];
      s = fmaf(wf[0], x0.x, s);
      s = fmaf(wf[1], x0.y, s);
      s = fmaf(wf[2], x0.z, s);
      s = fmaf(wf[3], x0.w, s);
      s = fmaf(wf[4], x1.x, s);
      s = fmaf(wf[5], x1.y, s);
      s = fmaf(wf[6], x1.z, s);
      s = fmaf(wf[7], x1.w, s);
      acc[b] = s;
    }
  }
}

// Fused decode-GEMV. Block = (row block rb, k-part kp); its waves take the
// column blocks of [kp*C, min(CB, (kp+1)*C)) in turn. Region per wave:
// stream columns, raw plane, activation slice.
template <int B, bool XBF16>
__global__ void __launch_bounds__(1024) gemv_kernel(GemvArgs p) {
  const GroupArgs& a = p.g;
  const uint32_t lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t waves = blockDim.x >> 6;
  const uint32_t S = a.S;
  const uint32_t per_wave = a.col_rows * kCol + 16 * S + p.x_words;
  uint32_t* cols = s_dyn + wave * per_wave;
  uint32_t* raw_lds = cols + a.col_rows * kCol;
  uint32_t* xs = raw_lds + 16 * S;
  const uint32_t sc_off = wave * per_wave + lane;
  const uint32_t* sc = s_dyn + sc_off;
  const uint32_t jmax = a.col_rows - 3;

  const uint32_t rb = blockIdx.x / p.KS, kp = blockIdx.x % p.KS;
  const uint32_t r0 = rb * a.GR;
  const uint32_t G = min(a.GR, a.rows - r0);
  const uint32_t N = G * a.GC;
  const uint32_t ldx = a.GC * S;  // slice row length
  const uint32_t* xl = xs + (XBF16 ? (lane / G) * (S / 2) : (lane / G) * S);
  const uint32_t cb_end = min(a.CB, (kp + 1) * p.C);
  uint32_t cb = kp * p.C + wave;
  Meta m;
  if (cb < cb_end) m = load_meta(a, rb * a.CB + cb, lane);
  load_tables(a.lut);
  __syncthreads();

  float acc[B];
#pragma unroll
  for (int b = 0; b < B; ++b) acc[b] = 0.f;

  for (; cb < cb_end; cb += waves) {
    uint32_t pos2 = issue_stream(a, cols, m, lane);
    issue_raw(a, raw_lds, m, lane);
    issue_x<B, XBF16>(p, xs, m.c0, lane);
    if (cb + waves < cb_end) {
      m = load_meta(a, rb * a.CB + cb + waves, lane);
      wait_vm1();
    } else {
      wait_vm0();
    }
    wave_sync_lds();
    if (lane < N) {
      const uint2* rl = reinterpret_cast<const uint2*>(raw_lds) + lane;
      for (uint32_t t = 0; t < S; t += 8) {
        const uint2 rw = rl[(t >> 3) * N];
        uint32_t e[8];
        decode8(sc, sc_off, jmax, pos2, e);
        mac8<B, XBF16>(acc, e, rw, xl, ldx, t);
      }
    }
    wait_lgkm0();
    wave_sync_lds();
  }
  // Reduction in a fixed order (the wave regions are free now): across waves
  // per lane, then across the GC lanes of each row.
  __syncthreads();
  float* red = reinterpret_cast<float*>(s_dyn);
#pragma unroll
  for (int b = 0; b < B; ++b) red[(wave * B + b) * 64 + lane] = acc[b];
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int b = 0; b < B; ++b) {
    float t = red[b * 64 + lane];
    for (uint32_t v = 1; v < waves; ++v) t += red[(v * B + b) * 64 + lane];
    red[b * 64 + lane] = t;
  }
  wait_lgkm0();
  wave_sync_lds();
  float s[B];
#pragma unroll
  for (int b = 0; b < B; ++b) {
    float t = 0.f;
    if (lane < G)
      for (uint32_t j = 0; j < a.GC; ++j) t += red[b * 64 + j * G + lane];
    s[b] = t;
  }
  const uint32_t ldy = a.rows;
  if (p.KS == 1) {
    if (lane < G)
#pragma unroll
      for (int b = 0; b < B; ++b) p.y[(uint64_t)b * ldy + r0 + lane] = s[b];
    return;
  }
  // Several blocks share this row block: publish the partial sums, and the
  // last block to arrive adds them in k-part order and resets the counter.
  // Partials are written and read with agent-scope atomics; the counter
  // increment is an agent-scope acquire-release, so the parts stored before
  // it (release) are visible to the block that sees the last count
  // (acquire, then a fence for the lanes that did not take part in it).
  const uint32_t ldp = a.RB * a.GR;
  if (lane < G)
#pragma unroll
    for (int b = 0; b < B; ++b)
      __hip_atomic_store(p.partial + ((uint64_t)kp * B + b) * ldp + r0 + lane, s[b], __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");  // every lane's parts, before the count
  uint32_t old = 0;
  if (lane == 0) old = __hip_atomic_fetch_add(p.counter + rb, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
  old = __shfl(old, 0, 64);
  if (old != p.KS - 1) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");  // every lane reads the parts published before the count
  if (lane < G) {
#pragma unroll
    for (int b = 0; b < B; ++b) {
      float t = 0.f;
      for (uint32_t k = 0; k < p.KS; ++k)
        t += __hip_atomic_load(p.partial + ((uint64_t)k * B + b) * ldp + r0 + lane, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
      p.y[(uint64_t)b * ldy + r0 + lane] = t;
    }
  }
  if (lane == 0) __hip_atomic_store(p.counter + rb, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------------------------------ fused GEMV on matrix cores

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// Sum of the waves' 16x16 accumulators and the output (fixed order), for the
// matrix-core kernels; `red` is LDS free for 16 floats per lane per wave.
__device__ inline void mfma_finish(const GemvArgs& p, const f32x4_t& acc, float* red, uint32_t wave,
                                   uint32_t waves, uint32_t lane, uint32_t rb, uint32_t kp, uint32_t r0,
                                   uint32_t G) {
  const GroupArgs& a = p.g;
  const uint32_t i = lane & 15, q = lane >> 4;
  __syncthreads();
#pragma unroll
  for (int v = 0; v < 4; ++v) red[(wave * 4 + v) * 64 + lane] = acc[v];
  __syncthreads();
  const uint32_t n = i, ldy = a.rows;
  const bool nb_ok = n < p.B;
  if (p.KS == 1) {
    // waves 0..3 each finish one of the four values of every lane (a block
    // of fewer waves: wave w finishes values w, w + waves, ...)
    for (uint32_t v = wave; v < 4; v += waves) {
      float t = red[v * 64 + lane];
      for (uint32_t w = 1; w < waves; ++w) t += red[(w * 4 + v) * 64 + lane];
      if (nb_ok && 4 * q + v < G) p.y[(uint64_t)n * ldy + r0 + 4 * q + v] = t;
    }
    return;
  }
  if (wave != 0) return;
  float s[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    float t = red[v * 64 + lane];
    for (uint32_t w = 1; w < waves; ++w) t += red[(w * 4 + v) * 64 + lane];
    s[v] = t;
  }
  // Split over column blocks: the same protocol as the vector kernel.
  const uint32_t ldp = a.RB * 16;
  if (nb_ok)
#pragma unroll
    for (int v = 0; v < 4; ++v)
      if (4 * q + v < G)
        __hip_atomic_store(p.partial + ((uint64_t)kp * p.B + n) * ldp + r0 + 4 * q + v, s[v], __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");  // every lane's parts, before the count
  uint32_t old = 0;
  if (lane == 0) old = __hip_atomic_fetch_add(p.counter + rb, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
  old = __shfl(old, 0, 64);
  if (old != p.KS - 1) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");  // every lane reads the parts published before the count
  if (nb_ok) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      if (4 * q + v >= G) continue;
      float t = 0.f;
      for (uint32_t k = 0; k < p.KS; ++k)
        t += __hip_atomic_load(p.partial + ((uint64_t)k * p.B + n) * ldp + r0 + 4 * q + v, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
      p.y[(uint64_t)n * ldy + r0 + 4 * q + v] = t;
    }
  }
  if (lane == 0) __hip_atomic_store(p.counter + rb, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Fused decode-GEMV for 16-row groups (GR = 16, GC = 4) and bf16 x, on the
// 16x16x32 bf16 matrix instruction. A group is exactly one A operand per
// 8-weight step: lane l = 16q + i decodes row r0 + i of column segment c0 + q,
// and its 8 weights are A[i][8q .. 8q+8); lane l also holds the activations
// x[n = i][(c0 + q)*S + t .. +8) as B[8q .. 8q+8][n]. The product sums the
// four segments' 8-weight pieces into C[row][n] (lane l: rows 4q .. 4q+3,
// batch i). Batch rows past B and rows past the block's G repeat valid data
// and are never written.
//
// Only the stream goes through LDS (DMA into lane columns); raw bytes and x
// are read straight into registers, KP steps ahead of their use, the last
// chunk of a group prefetching the next group's first chunk. SP = S/8 steps
// per group, unrolled so that every wait on a prefetch is exact.
template <int SP, bool XT>
__global__ void __launch_bounds__(1024) gemv_mfma_kernel(GemvArgs p) {
  constexpr int KP = SP < 8 ? SP : SP == 8 ? 8 : 4;  // 16 steps at depth 8 exceed 128 VGPRs
  const GroupArgs& a = p.g;
  const uint32_t lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t waves = blockDim.x >> 6;
  constexpr uint32_t S = SP * 8;
  const uint32_t per_wave = a.col_rows * kCol;
  uint32_t* cols = s_dyn + wave * per_wave;
  const uint32_t jmax = a.col_rows - 3;

  const uint32_t rb = blockIdx.x / p.KS, kp = blockIdx.x % p.KS;
  const uint32_t r0 = rb * 16;
  const uint32_t G = min(16u, a.rows - r0);
  const uint32_t N = G * 4;
  const uint32_t i = lane & 15, q = lane >> 4;
  const uint32_t mu = q * G + min(i, G - 1);  // the segment this lane decodes
  const uint32_t sc_off = wave * per_wave + mu;
  const uint32_t* sc = s_dyn + sc_off;
  const uint32_t rstride = N * 8;  // bytes between 8-weight steps of the raw plane
  // the lane's activations: x[n = i][(c0 + q)*S + 8k .. +8) at xlane + c0*XSEG + k*XSTEP (bytes), from x
  // itself or (XT) from its tiled copy, where the 16 batch rows' pieces of one
  // 8-column chunk are 256 contiguous bytes
  constexpr uint32_t XSEG = XT ? SP * 256 : S * 2, XSTEP = XT ? 256 : 16;
  const uint8_t* xlane = reinterpret_cast<const uint8_t*>(p.x) +
                         (XT ? (q * SP * 16 + i) * 16u : ((uint64_t)min(i, p.B - 1) * a.cols + q * S) * 2u);

  const uint32_t cb_end = min(a.CB, (kp + 1) * p.C);
  uint32_t cb = kp * p.C + wave;
  // Prologue: the first two groups' metadata and the table copy; once the
  // metadata is in, the first group's stream is copied to LDS and its raw
  // bytes and activations are requested behind it. The decode starts when the
  // table and the stream are in (the raw bytes of a step are waited for at
  // that step's product). All loads are unconditional (a wave without a
  // group reads its block's last group and discards it), so that no merge of
  // paths makes the compiler wait early.
  const uint32_t cb0 = min(cb, a.CB - 1);
  Meta m = load_meta(a, rb * a.CB + cb0, lane);
  Meta mn = load_meta(a, rb * a.CB + (cb + waves < cb_end ? cb + waves : cb0), lane);
  table_dma(a.lut);
  uint32_t pos2 = issue_stream(a, cols, m, lane);
  uint2 rw[KP];
  uint4 xv[KP];
  {
    const uint8_t* r = a.raw + m.first * S + mu * 8;
    const uint8_t* x = xlane + m.c0 * XSEG;
#pragma unroll
    for (int k = 0; k < KP; ++k) {
      rw[k] = *reinterpret_cast<const uint2*>(r + k * rstride);
      xv[k] = *reinterpret_cast<const uint4*>(x + k * XSTEP);
    }
  }
  // everything but the 2*KP raw and activation loads: the table and stream copies
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(2 * KP));
  asm volatile("" ::: "memory");
  __syncthreads();

  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
  for (; cb < cb_end; cb += waves) {
    // Group cb's stream is in the wave's columns; mn is the next group's metadata.
    const Meta cur = m;
    const bool more = cb + waves < cb_end;
    wave_sync_lds();
    const uint32_t pos2l = (uint32_t)__shfl((int)pos2, (int)mu, 64);
    const uint8_t* rcur = a.raw + cur.first * S + mu * 8;
    const uint8_t* xcur = xlane + cur.c0 * XSEG;
    // Prefetch source of the last chunk: the next group; after the wave's
    // last group, the lane's own first activation chunk (cache-resident) at
    // stride 0, so that the pipeline's loads stay unconditional without
    // reading HBM again.
    const uint8_t* rnext = more ? a.raw + mn.first * S + mu * 8 : reinterpret_cast<const uint8_t*>(xcur);
    const uint8_t* xnext = more ? xlane + mn.c0 * XSEG : xcur;
    const uint32_t rs_last = more ? rstride : 0u, xs_last = more ? XSTEP : 0u;
    uint32_t pd = pos2l;
#pragma unroll
    for (int t0 = 0; t0 < SP; t0 += KP) {
      const bool last = t0 + KP == SP;
      const uint8_t* rp = last ? rnext : rcur + (t0 + KP) * rstride;
      const uint8_t* xp = last ? xnext : xcur + (t0 + KP) * XSTEP;
      const uint32_t rs = last ? rs_last : rstride, xs = last ? xs_last : XSTEP;
#pragma unroll
      for (int k = 0; k < KP; ++k) {
        uint32_t e[8];
        decode8(sc, sc_off, jmax, pd, e);
        uint4 wv;
        wv.x = pack_pair(rw[k].x, 0, e[0], e[1]);
        wv.y = pack_pair(rw[k].x, 2, e[2], e[3]);
        wv.z = pack_pair(rw[k].y, 0, e[4], e[5]);
        wv.w = pack_pair(rw[k].y, 2, e[6], e[7]);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wv),
                                                      __builtin_bit_cast(bf16x8_t, xv[k]), acc, 0, 0, 0);
        mfma_operand_guard();
        rw[k] = *reinterpret_cast<const uint2*>(rp + k * rs);
        xv[k] = *reinterpret_cast<const uint4*>(xp + k * xs);
      }
    }
    wait_lgkm0();
    wave_sync_lds();
    if (more) {
      // the group after next's metadata, then the next group's stream copy
      m = mn;
      mn = load_meta(a, rb * a.CB + (cb + 2 * waves < cb_end ? cb + 2 * waves : cb + waves), lane);
      pos2 = issue_stream(a, cols, m, lane);
      wait_vm0();  // that copy (and the prefetches before it)
    }
  }
  wait_vm0();  // prefetches past the last group
  // Sum over waves in a fixed order (the wave regions are free now).
  mfma_finish(p, acc, reinterpret_cast<float*>(s_dyn), wave, waves, lane, rb, kp, r0, G);
}

// ------------------------------------------------------------------ batched decode-GEMM (prefill)

struct GemmArgs {
  GroupArgs g;
  const uint16_t* x;  // bf16 [T][cols]
  float* y;           // [T][rows]
  float* partial;     // workspace: KS x T x rows partial sums (KS > 1)
  uint32_t T;         // tokens
  uint32_t RS;        // row sets (16 row blocks each, one per wave)
  uint32_t KS;        // column-block ranges (blocks per row set and chunk)
  uint32_t cpb;       // column blocks per range
  uint32_t x_off;     // byte offset of the stream columns after the activation slice
};

// Activation slice in LDS: 16*NT token rows of 4*S bf16 (one column block),
// 16-byte chunk c of row r stored at chunk c ^ (r & 15), so that the 16 token
// rows a matrix-instruction operand reads fall in 16 different bank groups.
template <int SP>
__device__ inline uint32_t xslice_offset(uint32_t row, uint32_t chunk) {
  constexpr uint32_t kRowBytes = 4 * SP * 8 * 2;
  return row * kRowBytes + ((chunk ^ (row & 15)) << 4);
}

// Y[n][r] = sum_k W[r][k] X[n][k] for many tokens n (prefill). Block (ks, rs,
// ck): the column blocks ks*cpb .. of the 16 row blocks of row set rs (wave
// w: row block 16*rs + w), tokens 16*NT*ck .. of chunk ck, in NT tiles of 16.
// Per column block the block stages its activations once in LDS, shared by
// the waves, and each wave decodes its group step by step: each decoded
// 8-weight step (the A operand of the 16x16x32 bf16 matrix instruction, as in
// the GEMV) is multiplied with the NT token tiles (B operands from LDS). With
// one range (KS = 1) the block writes Y; otherwise it writes its partial sums
// and gemm_reduce_kernel adds the ranges in order (results do not vary
// between runs).
template <int SP, int NT>
__global__ void __launch_bounds__(1024) gemm_mfma_kernel(GemmArgs p) {
  constexpr uint32_t S = SP * 8;
  constexpr uint32_t kChunks = 4 * S / 8;       // 16-byte chunks per token row
  constexpr uint32_t kRows = 16 * NT;           // token rows of the slice
  constexpr uint32_t kCopies = kRows * kChunks / 64;
  const GroupArgs& a = p.g;
  const uint32_t lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t waves = blockDim.x >> 6;
  const uint32_t ks = blockIdx.x % p.KS;
  const uint32_t rest = blockIdx.x / p.KS;
  const uint32_t rs = rest % p.RS, ck = rest / p.RS;
  const uint32_t rb = min(rs * 16 + wave, a.RB - 1);  // waves past the last row block repeat it
  const bool own = rs * 16 + wave < a.RB;
  const uint32_t t0 = ck * kRows;
  const uint32_t r0 = rb * 16;
  const uint32_t G = min(16u, a.rows - r0);
  const uint32_t i = lane & 15, q = lane >> 4;
  const uint32_t mu = q * G + min(i, G - 1);
  uint8_t* xs = reinterpret_cast<uint8_t*>(s_dyn);
  const uint32_t per_wave = a.col_rows * kCol;
  const uint32_t col_base = p.x_off / 4 + wave * per_wave;
  uint32_t* cols = s_dyn + col_base;
  const uint32_t sc_off = col_base + mu;
  const uint32_t* sc = s_dyn + sc_off;
  const uint32_t jmax = a.col_rows - 3;
  const uint32_t rstride = G * 4 * 8;
  const uint32_t kb0 = ks * p.cpb, kb1 = min(a.CB, kb0 + p.cpb);

  f32x4_t acc[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (uint32_t cb = kb0; cb < kb1; ++cb) {
    if (cb != kb0) block_sync_lds();  // every wave is done with the slice and its columns
    // Metadata and raw bytes of all steps, then the table, stream and
    // activation copies into LDS.
    Meta m = load_meta(a, rb * a.CB + cb, lane);
    uint2 rw[SP];
    {
      const uint8_t* r = a.raw + m.first * S + mu * 8;
#pragma unroll
      for (int k = 0; k < SP; ++k) rw[k] = *reinterpret_cast<const uint2*>(r + k * rstride);
    }
    asm volatile("" : "+v"(m.nbw), "+v"(m.u0)::"memory");
    if (cb == kb0) table_dma(a.lut);
    const uint32_t pos2 = issue_stream(a, cols, m, lane);
    // Copy k of a wave fills the 1 KB at k*1024 of the slice; its lane L
    // writes position L there and so loads the chunk that the swizzle puts
    // at that position.
    for (uint32_t k = wave; k < kCopies; k += waves) {
      const uint32_t pos = k * 64 + lane;
      const uint32_t row = pos / kChunks, d = pos % kChunks;
      const uint32_t tok = min(t0 + row, p.T - 1);
      dma16(p.x + (uint64_t)tok * a.cols + cb * 4 * S + (d ^ (row & 15)) * 8,
            reinterpret_cast<uint32_t*>(xs + k * 1024));
    }
    wait_vm0();
    __syncthreads();

    uint32_t pd = (uint32_t)__shfl((int)pos2, (int)mu, 64);
#pragma unroll
    for (int k = 0; k < SP; ++k) {
      uint32_t e[8];
      decode8(sc, sc_off, jmax, pd, e);
      uint4 wv;
      wv.x = pack_pair(rw[k].x, 0, e[0], e[1]);
      wv.y = pack_pair(rw[k].x, 2, e[2], e[3]);
      wv.z = pack_pair(rw[k].y, 0, e[4], e[5]);
      wv.w = pack_pair(rw[k].y, 2, e[6], e[7]);
      const bf16x8_t A = __builtin_bit_cast(bf16x8_t, wv);
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const uint4 xb = *reinterpret_cast<const uint4*>(xs + xslice_offset<SP>(16 * j + i, q * SP + k));
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, __builtin_bit_cast(bf16x8_t, xb), acc[j], 0, 0, 0);
        mfma_operand_guard();
      }
    }
  }
  if (!own) return;
  // lane (q, i) holds rows 4q..4q+3 of token 16j + i of tile j
  const uint32_t R = a.rows;
  float* out = p.KS == 1 ? p.y : p.partial + (uint64_t)ks * p.T * R;
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    const uint32_t tok = t0 + 16 * j + i;
    if (tok >= p.T) continue;
    float* dst = out + (uint64_t)tok * R + r0 + 4 * q;
#pragma unroll
    for (int v = 0; v < 4; ++v)
      if (4 * q + v < G) dst[v] = acc[j][v];
  }
}

// Y = the sum of the KS partial products, in range order.
__global__ void __launch_bounds__(256) gemm_reduce_kernel(const float* partial, float* y, uint32_t KS,
                                                          uint64_t n) {
  for (uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n; k += (uint64_t)gridDim.x * blockDim.x) {
    float s = partial[k];
    for (uint32_t r = 1; r < KS; ++r) s += partial[(uint64_t)r * n + k];
    y[k] = s;
  }
}

// Tiled copy of bf16 activations for batches above one: xt[c][n][0..8) =
// x[min(n, B - 1)][8c .. 8c + 8) for the R = 16 rows n of a matrix-instruction
// B operand (or 32, 64: two or four of them, one after another), so that the
// 16 lanes reading one 8-column chunk read 256 contiguous bytes (from x itself
// they touch 16 rows, 16 cache lines).
template <uint32_t R>
__global__ void __launch_bounds__(256) xtile_kernel(const uint4* x, uint32_t B, uint32_t chunks, uint4* xt) {
  const uint32_t k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= chunks * R) return;
  const uint32_t c = k / R, n = min(k % R, B - 1);
  xt[k] = x[(uint64_t)n * chunks + c];
}

// ------------------------------------------------------------------ float16 format

// Decode tables of the float16 {1,5,5,5} format. Its kernels use no static
// LDS: the tables sit at the start of the dynamic LDS, the wave regions after.
// One table per field, in the order ml, e, mh, each indexed by an L-bit
// window (bit 0 first) with L the field's longest code (0 for a one-symbol
// field: one entry), so a complete code matches every window:
//   ml: code length in bits 0..3, ml in bits 16..20;
//   e:  length, e in bits 26..30;
//   mh: length, mh in bits 21..25;
// then the canonical tables of ml, e and mh in the aux format, for the
// bit-serial path. ORing a weight's three entries gives its bits 0..14 in
// bits 16..30. Sizing each table by its field's longest code keeps them small
// (the near-uniform mh field has 5-bit codes: 32 entries), which leaves LDS
// for 16 waves and spreads fewer distinct table words over the banks.
// Joint tables of two fields would save a read per weight, but subnormal and
// outlier weights carry two long codes at once (a pair past 13 bits in about
// one weight in 500); at 64 lanes x 8 weights per step that would send most
// steps through a slow path, and one table per field never needs one on such
// data. Two weights (at most 72 code bits) are decoded per 64-bit window,
// which holds 62 new bits; the rare pair longer than that (or a damaged code,
// whose entry is kEsc16 = 256) sends the lane through the bit-serial path. In
// the fast loop a position accumulates whole entries: bits 0..15 are the
// position (a column holds fewer than 2^16 bits), the weight bits pile up
// above.
constexpr int kLut16MaxBits = 12;
constexpr int kAux16Words = 3 * kAuxField;
constexpr uint32_t kTab16MaxWords = 3 * (1u << kLut16MaxBits) + kAux16Words;
constexpr uint32_t kEsc16 = 0x100u;
constexpr uint32_t kPosMask16 = 0xFFFFu;
constexpr uint32_t kAuxMl = 0, kAuxE = kAuxField, kAuxMh = 2 * kAuxField;

static_assert(HL_LUT_BYTES == kTab16MaxWords * 4, "the table buffer holds the largest format's tables");

// LDS layout of the float16 tables of one codebook (the same on the host,
// which builds them, and in the kernels, which read them).
struct Tab16 {
  uint32_t bits[3], base[3], aux, words;  // per field (ml, e, mh): window bits, word offset
};

static Tab16 tab16_layout(const hl_codebook16& cb) {
  Tab16 t;
  const hl_field_code5* f[3] = {&cb.ml, &cb.e, &cb.mh};
  uint32_t off = 0;
  for (int k = 0; k < 3; ++k) {
    uint32_t L = 0;
    if (f[k]->nsym > 1)
      for (int s = 0; s < 32; ++s) L = std::max<uint32_t>(L, f[k]->len[s]);
    t.bits[k] = L;
    t.base[k] = off;
    off += 1u << L;
  }
  t.aux = off;
  t.words = (off + kAux16Words + 3) & ~3u;
  return t;
}

struct Aux16 {
  uint32_t w[kAux16Words];
};

static Aux16 make_aux16(const hl_codebook16& cb) {
  Aux16 a;
  std::memset(&a, 0, sizeof(a));
  fill_aux_field(a.w + kAuxMl, cb.ml.len, 32, cb.ml.nsym, cb.ml.single);
  fill_aux_field(a.w + kAuxE, cb.e.len, 32, cb.e.nsym, cb.e.single);
  fill_aux_field(a.w + kAuxMh, cb.mh.len, 32, cb.mh.nsym, cb.mh.single);
  return a;
}

__global__ void __launch_bounds__(256) lut16_kernel(uint32_t* lut, Aux16 aux, Tab16 lay) {
  const uint32_t auxoff[3] = {kAuxMl, kAuxE, kAuxMh}, shift[3] = {16, 26, 21};
  for (int f = 0; f < 3; ++f) {
    const uint32_t n = 1u << lay.bits[f];
    for (uint32_t v = threadIdx.x; v < n; v += blockDim.x) {
      uint32_t u = 0;
      const int sym = field_from_bits(aux.w + auxoff[f], v, lay.bits[f], &u);
      lut[lay.base[f] + v] = sym < 0 ? kEsc16 : (u | ((uint32_t)sym << shift[f]));
    }
  }
  for (uint32_t i = lay.aux + threadIdx.x; i < lay.words; i += blockDim.x)
    lut[i] = i - lay.aux < (uint32_t)kAux16Words ? aux.w[i - lay.aux] : 0u;
}

// Copies the float16 tables to the start of the dynamic LDS (16-byte pieces
// through registers; kernels that wait on nothing else).
__device__ inline void load_tables16(const GroupArgs& a) {
  const uint32_t nv = a.t16_words / 4;
  const uint4* src = reinterpret_cast<const uint4*>(a.lut);
  uint4* dst = reinterpret_cast<uint4*>(s_dyn);
  for (uint32_t k = threadIdx.x; k < nv; k += blockDim.x) dst[k] = src[k];
}

// The same copy as direct global-to-LDS transfers (the caller waits, vmcnt).
__device__ inline void table16_dma(const GroupArgs& a) {
  const uint32_t nv = a.t16_words / 4;
  const uint32_t n = blockDim.x, w0 = threadIdx.x & ~63u, lane = threadIdx.x & 63;
  for (uint32_t k0 = w0; k0 < nv; k0 += n)
    if (k0 + lane < nv) dma16(a.lut + (k0 + lane) * 4, s_dyn + k0 * 4);
}

// Entry of field f's table for the window w (its index at bits 2.. of w).
template <int F>
__device__ inline uint32_t tab16(const GroupArgs& a, uint32_t w) {
  return *reinterpret_cast<const uint32_t*>(reinterpret_cast<const uint8_t*>(s_dyn) + a.t16_base[F] +
                                            (w & a.t16_mask[F]));
}

// 64-bit window of column bits [pos2, pos2 + 64), positions read through kPosMask16.
__device__ inline uint64_t load_window16(const uint32_t* sc, uint32_t pos2, uint32_t jmax) {
  const uint32_t j = min((pos2 & kPosMask16) >> 5, jmax);
  const uint32_t a = col_word(sc, j), b = col_word(sc, j + 1), c = col_word(sc, j + 2);
  return ((uint64_t)__builtin_amdgcn_alignbit(c, b, pos2) << 32) | __builtin_amdgcn_alignbit(b, a, pos2);
}

// Two weights from one 64-bit window: h[0..1] = weight bits 0..14 in bits
// 16..30 (other bits meaningless); p advanced by the six whole entries; flag
// collects the window's consumption plus one (bit 6 or above set: the two
// weights did not fit, or an escape).
__device__ inline void decode2_f16(const GroupArgs& a, const uint32_t* sc, uint32_t jmax, uint32_t& p,
                                   uint32_t& flag, uint32_t* h) {
  uint64_t W = load_window16(sc, p, jmax);
  uint32_t t[6];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    t[3 * k] = tab16<0>(a, (uint32_t)W);
    W = shift_window(W, t[3 * k]);
    t[3 * k + 1] = tab16<1>(a, (uint32_t)W);
    W = shift_window(W, t[3 * k + 1]);
    t[3 * k + 2] = tab16<2>(a, (uint32_t)W);
    if (k == 0) W = shift_window(W, t[2]);
  }
  const uint32_t used = t[0] + t[1] + t[2] + t[3] + t[4] + t[5];
  flag |= used + 1;
  p += used;
  h[0] = t[0] | t[1] | t[2];
  h[1] = t[3] | t[4] | t[5];
}

struct Dec8 {
  uint32_t pos2, h[8];
};

// Careful path of the float16 format: eight weights, each field decoded
// bit-serially (code(ml), code(e), code(mh)); pos2 clean (no weight bits
// above bit 15).
__device__ __attribute__((always_inline)) inline Dec8 decode8_f16_careful_body(uint32_t sc_off, uint32_t jmax,
                                                                               uint32_t pos2, uint32_t aux_off) {
  asm volatile("" ::: "memory");  // keeps its table reads inside the (cold) path
  const uint32_t* sc = s_dyn + sc_off;
  const uint32_t* aux = s_dyn + aux_off;
  Dec8 d;
  uint32_t p = pos2 + 2;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const uint32_t ml = slow_field(sc, aux + kAuxMl, p, jmax + 2);
    const uint32_t e = slow_field(sc, aux + kAuxE, p, jmax + 2);
    const uint32_t mh = slow_field(sc, aux + kAuxMh, p, jmax + 2);
    d.h[k] = (((e & 31) << 10) | ((mh & 31) << 5) | (ml & 31)) << 16;
  }
  d.pos2 = p - 2;
  return d;
}

__device__ __noinline__ Dec8 decode8_f16_careful(uint32_t sc_off, uint32_t jmax, uint32_t pos2, uint32_t aux_off) {
  return decode8_f16_careful_body(sc_off, jmax, pos2, aux_off);
}

// Eight float16 weights' bits 0..14 (in bits 16..30 of h[k]). A window that
// could not hold its two weights (or an escape) anywhere sends the lane
// through the careful path from the first of the eight; the fast entries read
// after it are discarded.
__device__ inline void decode8_f16(const GroupArgs& a, const uint32_t* sc, uint32_t sc_off, uint32_t jmax,
                                   uint32_t& pos2, uint32_t* h) {
  const uint32_t p0 = pos2;
  uint32_t p = p0, flag = 0;
  decode2_f16(a, sc, jmax, p, flag, h);
  decode2_f16(a, sc, jmax, p, flag, h + 2);
  decode2_f16(a, sc, jmax, p, flag, h + 4);
  decode2_f16(a, sc, jmax, p, flag, h + 6);
  if (__builtin_expect((flag & 0xFFC0u) != 0, 0)) {
    const Dec8 d = decode8_f16_careful(sc_off, jmax, p0 & kPosMask16, a.t16_aux);
    p = d.pos2;
#pragma unroll
    for (int k = 0; k < 8; ++k) h[k] = d.h[k];
  }
  pos2 = p;
}

// Eight float16 weights packed in pairs (weight 2m in the low half of dword
// m) from their decoded bits and the step's sign byte (bit k: weight k).
__device__ inline uint4 pack8_f16(const uint32_t* h, uint32_t sb) {
  uint32_t d[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const uint32_t v = __builtin_amdgcn_perm(h[2 * m + 1], h[2 * m], 0x07060302u) & 0x7FFF7FFFu;
    d[m] = v | (((sb >> (2 * m)) & 1u) << 15) | (((sb >> (2 * m + 1)) & 1u) << 31);
  }
  return uint4{d[0], d[1], d[2], d[3]};
}

// Decode to float16 bits; waves take groups in turn; region per wave: the
// stream columns. Signs are read straight from the sign plane.
__global__ void __launch_bounds__(1024) decode16_kernel(GroupArgs a, uint16_t* out) {
  const uint32_t lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t waves = blockDim.x >> 6;
  const uint32_t per_wave = a.col_rows * kCol;
  uint32_t* cols = s_dyn + a.t16_words + wave * per_wave;
  const uint32_t sc_off = a.t16_words + wave * per_wave + lane;
  const uint32_t* sc = s_dyn + sc_off;
  const uint32_t jmax = a.col_rows - 3;
  const uint32_t n_grp = a.RB * a.CB;
  const uint32_t stride = gridDim.x * waves;
  const uint32_t sb_per_seg = a.S / 8;
  uint32_t g = blockIdx.x * waves + wave;
  Meta m;
  if (g < n_grp) m = load_meta(a, g, lane);
  load_tables16(a);
  __syncthreads();
  for (; g < n_grp; g += stride) {
    uint32_t pos2 = issue_stream(a, cols, m, lane);
    const Meta cur = m;
    if (g + stride < n_grp) m = load_meta(a, g + stride, lane);
    wait_vm0();
    wave_sync_lds();
    if (lane < cur.N) {
      const uint32_t i = lane % cur.G, j = lane / cur.G;
      uint16_t* o = out + (uint64_t)(cur.r0 + i) * a.cols + (uint64_t)(cur.c0 + j) * a.S;
      const uint8_t* sg = a.raw + (cur.first + lane) * sb_per_seg;
      for (uint32_t t = 0; t < a.S; t += 8) {
        uint32_t h[8];
        decode8_f16(a, sc, sc_off, jmax, pos2, h);
        *reinterpret_cast<uint4*>(o + t) = pack8_f16(h, sg[t >> 3]);
      }
    }
    wait_lgkm0();
    wave_sync_lds();
  }
}

typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));

// The lane's sign bytes of one group (S/8 = SP bytes of its segment).
template <int SP>
struct Signs {
  uint4 v;
  __device__ inline void load(const uint8_t* p) {
    if constexpr (SP == 16) {
      v = *reinterpret_cast<const uint4*>(p);
    } else if constexpr (SP == 8) {
      const uint2 t = *reinterpret_cast<const uint2*>(p);
      v = uint4{t.x, t.y, 0u, 0u};
    } else if constexpr (SP == 4) {
      v = uint4{*reinterpret_cast<const uint32_t*>(p), 0u, 0u, 0u};
    } else if constexpr (SP == 2) {
      v = uint4{(uint32_t)*reinterpret_cast<const uint16_t*>(p), 0u, 0u, 0u};
    } else {
      v = uint4{(uint32_t)*p, 0u, 0u, 0u};
    }
  }
  __device__ inline uint32_t byte(int t) const {
    const uint32_t w = (t >> 2) == 0 ? v.x : (t >> 2) == 1 ? v.y : (t >> 2) == 2 ? v.z : v.w;
    return (w >> (8 * (t & 3))) & 0xFFu;
  }
};

// Fused decode-GEMV of the float16 format on the 16x16x32 float16 matrix
// instruction (16-row groups, float16 x): the bf16 matrix-core kernel's
// structure (lane 16q + i decodes row i of segment q; the A operand is its 8
// weights, the B operand x[n = i][8 activations]), with the float16 decode
// (two table reads per weight) and one sign load per lane and group.
template <int SP, bool XT>
__global__ void __launch_bounds__(1024) gemv16_mfma_kernel(GemvArgs p) {
  constexpr int KP = SP < 8 ? SP : SP == 8 ? 8 : 4;
  const GroupArgs& a = p.g;
  const uint32_t lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t waves = blockDim.x >> 6;
  constexpr uint32_t S = SP * 8;
  const uint32_t per_wave = a.col_rows * kCol;
  uint32_t* cols = s_dyn + a.t16_words + wave * per_wave;
  const uint32_t jmax = a.col_rows - 3;

  const uint32_t rb = blockIdx.x / p.KS, kp = blockIdx.x % p.KS;
  const uint32_t r0 = rb * 16;
  const uint32_t G = min(16u, a.rows - r0);
  const uint32_t i = lane & 15, q = lane >> 4;
  const uint32_t mu = q * G + min(i, G - 1);  // the segment this lane decodes
  const uint32_t sc_off = a.t16_words + wave * per_wave + mu;
  const uint32_t* sc = s_dyn + sc_off;
  // activations from x or (XT) from its tiled copy (see gemv_mfma_kernel)
  constexpr uint32_t XSEG = XT ? SP * 256 : S * 2, XSTEP = XT ? 256 : 16;
  const uint8_t* xlane = reinterpret_cast<const uint8_t*>(p.x) +
                         (XT ? (q * SP * 16 + i) * 16u : ((uint64_t)min(i, p.B - 1) * a.cols + q * S) * 2u);

  const uint32_t cb_end = min(a.CB, (kp + 1) * p.C);
  uint32_t cb = kp * p.C + wave;
  const uint32_t cb0 = min(cb, a.CB - 1);
  Meta m = load_meta(a, rb * a.CB + cb0, lane);
  Meta mn = load_meta(a, rb * a.CB + (cb + waves < cb_end ? cb + waves : cb0), lane);
  uint4 xv[KP];
  Signs<SP> sg;
  {
    const uint8_t* x = xlane + m.c0 * XSEG;
#pragma unroll
    for (int k = 0; k < KP; ++k) xv[k] = *reinterpret_cast<const uint4*>(x + k * XSTEP);
    sg.load(a.raw + (m.first + mu) * SP);
  }
  asm volatile("" : "+v"(m.nbw), "+v"(m.u0)::"memory");
  table16_dma(a);
  uint32_t pos2 = issue_stream(a, cols, m, lane);
  wait_vm0();
  __syncthreads();

  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
  for (; cb < cb_end; cb += waves) {
    const Meta cur = m;
    const bool more = cb + waves < cb_end;
    wait_vm0();
    wave_sync_lds();
    const uint32_t pos2l = (uint32_t)__shfl((int)pos2, (int)mu, 64);
    const uint8_t* xcur = xlane + cur.c0 * XSEG;
    const uint8_t* xnext = more ? xlane + mn.c0 * XSEG : xcur;
    const uint32_t xs_last = more ? XSTEP : 0u;
    const Signs<SP> sgc = sg;
    uint32_t pd = pos2l;
#pragma unroll
    for (int t0 = 0; t0 < SP; t0 += KP) {
      const bool last = t0 + KP == SP;
      const uint8_t* xp = last ? xnext : xcur + (t0 + KP) * XSTEP;
      const uint32_t xs = last ? xs_last : XSTEP;
#pragma unroll
      for (int k = 0; k < KP; ++k) {
        uint32_t h[8];
        decode8_f16(a, sc, sc_off, jmax, pd, h);
        const uint4 wv = pack8_f16(h, sgc.byte(t0 + k));
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, wv),
                                                     __builtin_bit_cast(f16x8_t, xv[k]), acc, 0, 0, 0);
        mfma_operand_guard();
        xv[k] = *reinterpret_cast<const uint4*>(xp + k * xs);
      }
    }
    wait_lgkm0();
    wave_sync_lds();
    if (more) {
      m = mn;
      mn = load_meta(a, rb * a.CB + (cb + 2 * waves < cb_end ? cb + 2 * waves : cb + waves), lane);
      pos2 = issue_stream(a, cols, m, lane);
      sg.load(a.raw + (m.first + mu) * SP);
    }
  }
  wait_vm0();  // prefetches past the last group
  mfma_finish(p, acc, reinterpret_cast<float*>(s_dyn + a.t16_words), wave, waves, lane, rb, kp, r0, G);
}

// ------------------------------------------------------------------ persistent fused GEMV

// Persistent form of the matrix-core kernel for S = 8*SP (SP = 4 or 8) and matrices with at
// least one 16-row block per block of the grid and at least as many column
// blocks as waves. Block b takes row blocks b, b + grid, ...; its waves take
// the row block's column blocks wave, wave + waves, ... The table is copied
// once per block. With DEC it decodes to bf16 instead (hl_decode): a lane
// keeps its segment's weights (S*2 bytes of one row) and stores them at the
// group's end, with no activations and no sums.
//
// While a wave decodes group k from its LDS columns, group k+1's stream words
// (JT per lane, four per load), raw bytes and activations are loaded into
// registers and group k+2's metadata arrives; after the decode the stream
// words are written to the columns. Only ordinary loads are in flight in the
// loop (no LDS copies, which the compiler does not order with them), so every
// wait the compiler places is exact. At a row block's end the waves add their
// accumulators through their columns in a fixed order (before the next
// group's words go in) and four waves write y.
// Arguments of the persistent kernel: up to kMaxParts matrices with the same
// columns and container geometry that share x (a grouped launch); blocks
// [part0[m], part0[m + 1]) work on matrix m and write y[m].
constexpr uint32_t kMaxParts = 4;
struct StreamArgs {
  GemvArgs p;  // x, batch (p.g and p.y unused)
  GroupArgs g[kMaxParts];
  float* y[kMaxParts];
  uint32_t part0[kMaxParts + 1];
  uint32_t n;
};

// One matrix (Args = GemvArgs), or a grouped launch (Args = StreamArgs: a
// block first finds its matrix, with a dependent load before its arguments;
// the one-matrix kernel keeps the small argument block and reads it at fixed
// places).
template <class Args>
__device__ inline const GemvArgs& gemv_args(const Args& x) {
  if constexpr (std::is_same_v<Args, StreamArgs>) return x.p; else return x;
}

// TB selects the decode table: 0 the joint table (bf16 formats), 1 the
// bounded-pair table (split format, pairs of at most kBpBits bits), 2 the
// float16 format's three field tables (at the start of the dynamic LDS, its
// sign plane instead of raw bytes, the float16 matrix instruction).
// NT = 16-token tiles of activations per matrix instruction step: 1 (up to 16
// activation rows), or 2 or 4 for prefill products of 17 to 32 or 33 to 64
// tokens (one bf16 matrix, activations from their tiled copy).
// Blocks of at most 16 waves (8 decoding, whose registers hold a group's
// weights until its stores, or with several tiles; 12 for the float16
// product, whose longer stream columns need more registers).
constexpr uint32_t stream_threads(bool dec, int tb, int nt = 1) {
  return dec || nt > 1 ? 512 : tb == 2 ? 768 : 1024;
}

template <int SP, int JT, bool XT, class Args, bool DEC, int TB, int NT = 1>
__global__ void __launch_bounds__(stream_threads(DEC, TB, NT)) gemv_stream_kernel(Args sa) {
  constexpr bool BP = TB == 1, F16 = TB == 2;
  constexpr uint32_t S = SP * 8;
  constexpr uint32_t kRows = JT + 1, kBuf = kRows * kCol;
  static_assert(JT % 4 == 0 && kBuf >= 256, "layout");
  static_assert(!(F16 && std::is_same_v<Args, StreamArgs>), "the float16 form runs one matrix per launch");
  static_assert(NT == 1 || ((NT == 2 || NT == 4) && XT && !DEC && !F16 && std::is_same_v<Args, GemvArgs> &&
                            kBuf >= 256u * NT),
                "several token tiles: one bf16 matrix, every tile's sums in a wave region");
  constexpr int NE = NT > 1 ? NT - 1 : 1;  // the tiles after the first (their arrays)
  constexpr bool kMulti = std::is_same_v<Args, StreamArgs>;
  const GemvArgs& p = gemv_args(sa);
  // this block's matrix (wave-uniform; its arguments are read in place)
  const GroupArgs* ap = &p.g;
  float* yp = p.y;
  uint32_t bid = blockIdx.x, nblk = gridDim.x;
  if constexpr (kMulti) {
    uint32_t m = 0;
    for (uint32_t k = 1; k < sa.n; ++k) m += blockIdx.x >= sa.part0[k] ? 1u : 0u;
    ap = &sa.g[m];
    yp = sa.y[m];
    bid = blockIdx.x - sa.part0[m];
    nblk = sa.part0[m + 1] - sa.part0[m];
  }
  const GroupArgs& a = *ap;
  uint16_t* const outp = reinterpret_cast<uint16_t*>(yp);  // decoding: the 16-bit output (GemvArgs::y)
  const uint32_t lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t waves = blockDim.x >> 6;
  const uint32_t kTab = F16 ? a.t16_words : 0u;  // dynamic LDS words before the wave regions
  uint32_t* cols = s_dyn + kTab + wave * kBuf;
  const uint32_t jmax = kRows - 3;
  const uint32_t i = lane & 15, q = lane >> 4;
  const uint32_t lane_off = (lane % kBpCopies) * 4;  // bounded pairs: the lane's table copy
  // byte offset of the lane's activations x[n = i][(c0 + q)*S + 8k .. +8) at
  // x + c0*XSEG + xoff + k*XSTEP, from x itself or (XT) from its tiled copy,
  // where the 16 batch rows' pieces of one 8-column chunk are 256 contiguous
  // bytes (a wave-uniform base plus a 32-bit lane offset lets the prefetch
  // loads address as scalar base + vector offset + immediate)
  // (NT tiles: 16 NT rows per chunk in the tiled copy, tile after tile)
  constexpr uint32_t XSEG = XT ? SP * 256 * NT : S * 2, XSTEP = XT ? 256 * NT : 16;
  const uint32_t xoff = XT ? (q * SP * 16 * NT + i) * 16u : (min(i, p.B - 1) * a.cols + q * S) * 2u;
  // tile u > 0: activation rows 16u + i, 256u bytes after the first tile's
  // in the tiled copy
  const uint8_t* xbytes = reinterpret_cast<const uint8_t*>(p.x);
  const uint32_t CB = a.CB, RB = a.RB, nj = (CB + waves - 1) / waves;
  const uint32_t last_group = RB * CB - 1;

  // the wave's groups in order: round t (row block bid + t*nblk of the
  // block's matrix), step j; branch-free (a branch between a load and its use
  // makes the compiler's wait for it conservative)
  auto rb_of = [&](uint32_t t) { return bid + t * nblk; };
  auto advance = [&](uint32_t& t, uint32_t& j) {
    const bool same = wave + (j + 1) * waves < CB;
    t = same ? t : t + 1;
    j = same ? j + 1 : 0u;
  };
  auto group = [&](uint32_t t, uint32_t j) { return min(rb_of(t) * CB + wave + j * waves, last_group); };
  auto lane_mu = [&](uint32_t rb) {
    const uint32_t G = min(16u, a.rows - rb * 16);
    return q * G + min(i, G - 1);
  };

  // Prologue. The table (bounded pairs: its entries into registers; else
  // the copy to LDS) and the first two groups' metadata are requested first;
  // the table entries are stored to LDS while the metadata is on its way.
  // Then the first group's stream words, and right behind them its raw bytes
  // and activations: the decode starts once the stream words are in (loads
  // return in order), and the raw bytes of a step are waited for only at that
  // step's product.
  uint32_t t1 = 0, j1 = 0;
  advance(t1, j1);
  const uint32_t g0 = group(0, 0);
  const uint32_t g1 = rb_of(t1) < RB ? group(t1, j1) : g0;
  uint32_t te[kBpPerThread];
  if constexpr (BP) bp_table_load(a.lut, te);
  else if constexpr (F16) table16_dma(a);
  else table_dma(a.lut);
  Meta m0 = load_meta(a, g0, lane);
  Meta m1 = load_meta(a, g1, lane);
  if constexpr (BP) bp_table_store(te);
  u32x4_a4 sw[JT / 4];
  uint32_t pos2 = stream_load<JT>(a, m0, lane, sw) - (BP ? kBpShift - 2 : 0u);
  uint2 rw[F16 ? 1 : SP];  // raw bytes of the next group's steps (bf16 formats)
  Signs<SP> sg, sgn;       // float16: the lane's sign bytes of this and the next group
  uint4 xv[SP];
  uint4 xe[NE][SP];  // the other tiles' activations
  // raw bytes of the first group's first half of the steps with its stream
  // words, the second half once those are in: every wave requests its first
  // group at once, and a wave's stream words would otherwise queue behind
  // the other waves' raw bytes for all eight steps
  constexpr int kEarlyRaw = F16 ? 0 : SP / 2;
  const uint8_t* raw0 = nullptr;
  {
    const uint32_t rb = g0 / CB;
    const uint32_t G = min(16u, a.rows - rb * 16);
    raw0 = a.raw + m0.first * S + lane_mu(rb) * 8;
    if constexpr (F16) sg.load(a.raw + (m0.first + lane_mu(rb)) * SP);
#pragma unroll
    for (int k = 0; k < SP; ++k) {
      if constexpr (!F16) if (k < kEarlyRaw) rw[k] = *reinterpret_cast<const uint2*>(raw0 + k * G * 32u);
      if constexpr (!DEC) xv[k] = *reinterpret_cast<const uint4*>(xbytes + m0.c0 * XSEG + xoff + k * XSTEP);
#pragma unroll
      for (int u = 1; u < NT; ++u)
        xe[u - 1][k] = *reinterpret_cast<const uint4*>(xbytes + m0.c0 * XSEG + xoff + 256u * u + k * XSTEP);
    }
    if constexpr (NT == 4) {
      // a precaution: no scalar write into these loads' scalar base right
      // behind them (such a write two instructions after a buffer load was
      // the one pattern of a form of this kernel that gave wrong products;
      // of the forms here only this one's prologue had it)
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("s_nop 2");
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  stream_store<JT>(cols, sw, lane);
  // everything but the raw (or sign) and activation loads
  constexpr int kRawLoads = F16 ? 1 : kEarlyRaw;
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(kRawLoads + (DEC ? 0 : SP * NT)));
  asm volatile("" ::: "memory");
  if constexpr (!F16) {
    const uint32_t G = min(16u, a.rows - (g0 / CB) * 16);
#pragma unroll
    for (int k = kEarlyRaw; k < SP; ++k) rw[k] = *reinterpret_cast<const uint2*>(raw0 + k * G * 32u);
  }
  __syncthreads();

  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
  f32x4_t acce[NE];  // the other tiles' sums
#pragma unroll
  for (int u = 0; u < NE; ++u) acce[u] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (uint32_t t = 0; rb_of(t) < RB; ++t) {
    const uint32_t rb = rb_of(t);
    const uint32_t G = min(16u, a.rows - rb * 16);
    const uint32_t mu = q * G + min(i, G - 1);
    const uint32_t sc_off = kTab + wave * kBuf + mu;
    const uint32_t* sc = s_dyn + sc_off;
    for (uint32_t j = 0; j < nj; ++j) {
      if (wave + j * waves >= CB) continue;
      // the next two groups of this wave
      uint32_t tn = t, jn = j;
      advance(tn, jn);
      const bool okn = rb_of(tn) < RB;
      uint32_t t2 = tn, j2 = jn;
      advance(t2, j2);
      const uint32_t g2 = rb_of(t2) < RB ? group(t2, j2) : group(t, j);
      const uint32_t rbn = okn ? rb_of(tn) : rb;
      const uint32_t Gn = min(16u, a.rows - rbn * 16);
      const uint64_t n_first = m1.first;
      const uint32_t n_c0 = m1.c0;
      // the next group's stream words (this group's again after the last),
      // then the metadata of the group after it
      uint32_t pos2n = stream_load<JT>(a, m1, lane, sw) - (BP ? kBpShift - 2 : 0u);
      m1 = load_meta(a, g2, lane);
      // prefetch source: the next group, else the lane's cached activations
      // (decoding: the current group's raw bytes)
      const uint32_t cur_c0 = (wave + j * waves) * 4;
      const uint8_t* rbase = okn    ? a.raw + n_first * S
                             : DEC ? a.raw + ((uint64_t)rb * 16u * a.L + (uint64_t)cur_c0 * G) * S
                                   : xbytes + cur_c0 * XSEG;
      const uint32_t roff = okn ? lane_mu(rbn) * 8 : DEC ? mu * 8 : xoff;
      const uint32_t rs = okn ? Gn * 32u : 0u;
      const uint8_t* xbase = xbytes + (okn ? n_c0 : cur_c0) * XSEG;
      uint32_t pd = (uint32_t)__shfl((int)pos2, (int)mu, 64);
      uint4 dv[DEC ? SP : 1];  // decoding: the lane's weights of the group
      // float16: the next group's sign bytes (after the wave's last group of
      // the launch, the plane's first bytes, discarded)
      const uint8_t* sgnext = okn ? a.raw + (n_first + lane_mu(rbn)) * SP : a.raw;
#pragma unroll
      for (int k = 0; k < SP; ++k) {
        uint4 wv;
        if constexpr (F16) {
          uint32_t h[8];
          decode8_f16(a, sc, sc_off, jmax, pd, h);
          wv = pack8_f16(h, sg.byte(k));
        } else {
          uint32_t e[8];
          if constexpr (BP) bp_decode8(sc, jmax, pd, e, lane_off); else decode8(sc, sc_off, jmax, pd, e);
          wv.x = pack_pair(rw[k].x, 0, e[0], e[1]);
          wv.y = pack_pair(rw[k].x, 2, e[2], e[3]);
          wv.z = pack_pair(rw[k].y, 0, e[4], e[5]);
          wv.w = pack_pair(rw[k].y, 2, e[6], e[7]);
        }
        if constexpr (DEC) {
          dv[k] = wv;
        } else {
          if constexpr (F16)
            acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, wv),
                                                         __builtin_bit_cast(f16x8_t, xv[k]), acc, 0, 0, 0);
          else if constexpr (NT == 1)
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wv),
                                                          __builtin_bit_cast(bf16x8_t, xv[k]), acc, 0, 0, 0);
          if constexpr (NT == 1) {
            mfma_operand_guard();
          } else {
            // several tiles: each matrix instruction directly followed by
            // its guard, in this order (left to the scheduler, the
            // instructions moved into the next step's decode, or the guard
            // between two of them, and a write to their operand registers
            // came right after)
            __builtin_amdgcn_sched_barrier(0);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wv),
                                                          __builtin_bit_cast(bf16x8_t, xv[k]), acc, 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
            mfma_operand_guard();
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int u = 0; u < NT - 1; ++u) {
              acce[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wv),
                                                                __builtin_bit_cast(bf16x8_t, xe[u][k]), acce[u], 0, 0,
                                                                0);
              __builtin_amdgcn_sched_barrier(0);
              mfma_operand_guard();
              __builtin_amdgcn_sched_barrier(0);
            }
          }
          // x first: the wait for the raw bytes at their use then covers both
          xv[k] = *reinterpret_cast<const uint4*>(xbase + xoff + k * XSTEP);
#pragma unroll
          for (int u = 1; u < NT; ++u)
            xe[u - 1][k] = *reinterpret_cast<const uint4*>(xbase + xoff + 256u * u + k * XSTEP);
        }
        if constexpr (F16) {
          if (k == 0) sgn.load(sgnext);
        } else {
          rw[k] = *reinterpret_cast<const uint2*>(rbase + k * rs + roff);
        }
      }
      if constexpr (F16) sg = sgn;
      if constexpr (DEC && F16) {
        // float16 (its decode already LDS-bound: the transposition below cost
        // 5% there): row r0 + i, columns (c0 + q)*S .. + S back to back
        if (i < G) {
          uint4* o = reinterpret_cast<uint4*>(outp + (uint64_t)(rb * 16 + i) * a.cols + (cur_c0 + q) * S);
#pragma unroll
          for (int k = 0; k < SP; ++k) o[k] = dv[k];
        }
      } else if constexpr (DEC) {
        // The group's 16 rows x 4 segments, transposed through the wave's
        // column region (its stream words are consumed), four rows at a time,
        // so that each store instruction writes whole output rows: 32 (S =
        // 64) or 16 lanes per row of 4 segments, 16 bytes each. Stored
        // straight from the lanes (row i, segment q: 16-byte chunks 128 or 64
        // bytes apart), every store instruction touched 64 cache lines:
        // 28672x8192 265 us against 170 us with whole rows (timing run).
        // Chunk kk of tile row m (= row * 4 + segment) sits in slot
        // kk ^ (m % SP) of that row, so that a write's lanes spread over the banks.
        constexpr uint32_t kLanesPerRow = 4 * SP, kRowsPerStore = 64 / kLanesPerRow, kPassRows = 4;
        uint4* tile = reinterpret_cast<uint4*>(cols);
        const uint32_t c = lane % kLanesPerRow, cq = c / SP, ck = c % SP;
        uint16_t* orow = outp + (uint64_t)(rb * 16) * a.cols + cur_c0 * S + c * 8;
#pragma unroll
        for (uint32_t h = 0; h < 16; h += kPassRows) {
          if (i - h < kPassRows) {
            const uint32_t m = (i - h) * 4 + q;
#pragma unroll
            for (int k = 0; k < SP; ++k) tile[m * SP + ((uint32_t)k ^ (m % SP))] = dv[k];
          }
          wait_lgkm0();
          wave_sync_lds();
#pragma unroll
          for (uint32_t r0 = 0; r0 < kPassRows; r0 += kRowsPerStore) {
            const uint32_t rr = r0 + lane / kLanesPerRow, m = rr * 4 + cq;
            const uint4 v = tile[m * SP + (ck ^ (m % SP))];
            if (h + rr < G) *reinterpret_cast<uint4*>(orow + (uint64_t)(h + rr) * a.cols) = v;
          }
          wait_lgkm0();
          wave_sync_lds();
        }
      }
      wait_lgkm0();
      wave_sync_lds();
      pos2 = pos2n;
      // the next group's words go in now, unless this was the wave's last
      // group of the row block (the columns first carry the row block's sum)
      if (okn && rb_of(tn) == rb) {
        stream_store<JT>(cols, sw, lane);
        wait_lgkm0();
        wave_sync_lds();
      }
    }
    // End of the row block: add the waves' accumulators in a fixed order
    // (LDS-only barriers: the loads in flight stay in flight).
    if constexpr (!DEC) {
      block_sync_lds();
      float* red = reinterpret_cast<float*>(cols);
#pragma unroll
      for (int v = 0; v < 4; ++v) red[v * 64 + lane] = acc[v];
      acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int u = 0; u < NT - 1; ++u) {
#pragma unroll
        for (int v = 0; v < 4; ++v) red[256 * (u + 1) + v * 64 + lane] = acce[u][v];
        acce[u] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      }
      block_sync_lds();
      if constexpr (NT == 1) {
        if (wave < 4) {
          const uint32_t v = wave;
          float sum = 0.f;
          for (uint32_t w = 0; w < waves; ++w) sum += reinterpret_cast<const float*>(s_dyn + kTab + w * kBuf)[v * 64 + lane];
          if (i < p.B && 4 * q + v < G) yp[(uint64_t)i * a.rows + rb * 16 + 4 * q + v] = sum;
        }
      } else {
        // wave u % waves sums piece v = u % 4 of tile u / 4 (blocks of 8 waves)
        for (uint32_t u = wave; u < 4u * NT; u += waves) {
          const uint32_t v = u & 3, tile = u >> 2, n = tile * 16 + i;
          float sum = 0.f;
          for (uint32_t w = 0; w < waves; ++w)
            sum += reinterpret_cast<const float*>(s_dyn + kTab + w * kBuf)[tile * 256 + v * 64 + lane];
          if (n < p.B && 4 * q + v < G) yp[(uint64_t)n * a.rows + rb * 16 + 4 * q + v] = sum;
        }
      }
      block_sync_lds();
    }
    // the next group's words, held back for the sum (none after the last
    // row block, which has no next group)
    if (rb_of(t + 1) < RB) {
      stream_store<JT>(cols, sw, lane);
      wait_lgkm0();
      wave_sync_lds();
    }
  }
  wait_vm0();  // prefetches past the last group
}

// ------------------------------------------------------------------ bf16 GEMV

// One wave per row; lanes stride the row in 8-weight chunks; dot2 on pairs.
template <int B, bool XBF16>
__global__ void __launch_bounds__(1024) gemv_bf16_kernel(const uint16_t* w, const void* x, float* y,
                                                        uint32_t rows, uint32_t cols) {
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t waves = blockDim.x >> 6;
  for (uint32_t r = blockIdx.x * waves + (threadIdx.x >> 6); r < rows; r += gridDim.x * waves) {
    float acc[B];
#pragma unroll
    for (int b = 0; b < B; ++b) acc[b] = 0.f;
    const uint16_t* wr = w + (uint64_t)r * cols;
    for (uint32_t c = lane * 8; c < cols; c += 512) {
      const uint4 wv = *reinterpret_cast<const uint4*>(wr + c);
#pragma unroll
      for (int b = 0; b < B; ++b) {
        if constexpr (XBF16) {
          const uint4 xv = *reinterpret_cast<const uint4*>(
              reinterpret_cast<const uint16_t*>(x) + (uint64_t)b * cols + c);
          float s = acc[b];
          s = dot2(wv.x, xv.x, s);
          s = dot2(wv.y, xv.y, s);
          s = dot2(wv.z, xv.z, s);
          s = dot2(wv.w, xv.w, s);
          acc[b] = s;
        } else {
          const float* xf = reinterpret_cast<const float*>(x) + (uint64_t)b * cols + c;
          const float4 x0 = *reinterpret_cast<const float4*>(xf);
          const float4 x1 = *reinterpret_cast<const float4*>(xf + 4);
          const uint32_t ww[4] = {wv.x, wv.y, wv.z, wv.w};
          const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
          float s = acc[b];
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            s = fmaf(__uint_as_float(ww[k] << 16), xs[2 * k], s);
            s = fmaf(__uint_as_float(ww[k] & 0xFFFF0000u), xs[2 * k + 1], s);
          }
          acc[b] = s;
        }
      }
    }
#pragma unroll
    for (int b = 0; b < B; ++b) {
      float s = acc[b];
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
      if (lane == 0) y[(uint64_t)b * rows + r] = s;
    }
  }
}

// ------------------------------------------------------------------ launch helpers

static int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return 256;
  return cus;
}

constexpr uint32_t kMaxLds = 160 * 1024;

struct Plan {
  GroupArgs ga;
  uint32_t waves;
  size_t lds;       // dynamic LDS: (float16 tables) + the wave regions
  size_t tab_dyn;   // bytes of the float16 tables in it
  size_t wave_bytes;  // bytes of one wave region
  // dynamic LDS of a block of w waves
  size_t lds_for(uint32_t w) const { return tab_dyn + (size_t)w * wave_bytes; }
};

static bool is_fp16(const hl_tensor* t) { return t->format == HL_FORMAT_FP16; }

// Rows of the stream columns: row 0 padding, the longest segment starting at
// bit 31 of row 1, three rows of window overrun (the bf16 decode reads four
// words at once).
static uint32_t col_rows_for(uint32_t max_seg_bits) { return 1 + ((31 + max_seg_bits + 31) >> 5) + 3; }

// raw_lds: the kernel stages the raw plane (64*S bytes per wave) in LDS.
static hl_status make_plan(const hl_tensor* t, uint32_t extra_words_per_wave, bool raw_lds, Plan* pl) {
  if (!t || !t->blob_dev || !t->lut_dev) return HL_EINVAL;
  if (t->rows >= (1ull << 31) || t->cols >= (1ull << 31) || t->n_grp >= (1ull << 31))
    return HL_EUNSUPPORTED;
  GroupArgs& a = pl->ga;
  std::memset(&a, 0, sizeof(a));
  const uint8_t* b = t->blob_dev;
  a.seg_len8 = b + t->off_seg_bits;
  a.grp_meta = reinterpret_cast<const uint32_t*>(b + t->off_grp_off);
  a.stream = reinterpret_cast<const uint4*>(b + t->off_stream);
  a.raw = b + t->off_raw;
  a.lut = t->lut_dev;
  a.rows = (uint32_t)t->rows;
  a.cols = (uint32_t)t->cols;
  a.S = t->seg_len;
  a.L = (uint32_t)(t->cols / t->seg_len);
  a.GR = t->grp_rows;
  a.GC = HL_GROUP_SEGS / t->grp_rows;
  a.CB = a.L / a.GC;
  a.RB = (uint32_t)((t->rows + a.GR - 1) / a.GR);
  a.stream_units = (uint32_t)std::min<uint64_t>((t->off_raw - t->off_stream) / 16, 0xFFFFFFFFu);
  a.max_units = t->max_grp_units;
  a.col_rows = col_rows_for(t->max_seg_bits);
  const uint32_t per_wave = a.col_rows * kCol + (raw_lds ? 16 * t->seg_len : 0) + extra_words_per_wave;
  // LDS: the tables (static for the bf16 formats, at the start of the
  // dynamic region for float16) plus one region per wave.
  if (is_fp16(t)) {
    const Tab16 lay = tab16_layout(t->cb16);
    for (int k = 0; k < 3; ++k) {
      a.t16_mask[k] = ((1u << lay.bits[k]) - 1) << 2;
      a.t16_base[k] = lay.base[k] * 4;
    }
    a.t16_aux = lay.aux;
    a.t16_words = lay.words;
  }
  const size_t tab_static = is_fp16(t) ? 0 : (size_t)(kLutN + kAuxWords) * 4;
  const size_t tab_dyn = is_fp16(t) ? (size_t)a.t16_words * 4 : 0;
  uint32_t waves = kMaxWaves;
  while (waves > 1 && tab_static + tab_dyn + (size_t)waves * per_wave * 4 > kMaxLds) --waves;
  const size_t lds = tab_dyn + (size_t)waves * per_wave * 4;
  if (tab_static + lds > kMaxLds) return HL_EUNSUPPORTED;
  pl->waves = waves;
  pl->lds = lds;
  pl->tab_dyn = tab_dyn;
  pl->wave_bytes = (size_t)per_wave * 4;
  return HL_OK;
}

template <class K, class... A>
static hl_status launch(K kernel, dim3 grid, dim3 block, size_t lds, hipStream_t s, A... args) {
  if (lds + (kLutN + kAuxWords) * 4 > 64 * 1024) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
      return HL_EHIP;
  }
  hipLaunchKernelGGL(kernel, grid, block, lds, s, args...);
  return hipGetLastError() == hipSuccess ? HL_OK : HL_EHIP;
}

template <int B>
static hl_status launch_gemv_b(bool xbf16, dim3 grid, dim3 block, size_t lds, hipStream_t s,
                               const GemvArgs& p) {
  return xbf16 ? launch(gemv_kernel<B, true>, grid, block, lds, s, p)
               : launch(gemv_kernel<B, false>, grid, block, lds, s, p);
}

// Stream words per lane the persistent kernel is built for (the smallest one
// not below the tensor's longest segment is used), per segment length.
static int stream_rows_for(uint32_t seg_len, uint32_t col_rows, bool f16) {
  // the float16 format's codes take about 10 bits per weight, the bf16
  // formats' about 4
  static const int kJT64[] = {12, 16, 20}, kJT32[] = {8, 12}, kJT64h[] = {24, 28, 32}, kJT32h[] = {12, 16};
  if (seg_len != 64 && seg_len != 32) return 0;
  const int* set = seg_len == 64 ? (f16 ? kJT64h : kJT64) : (f16 ? kJT32h : kJT32);
  const int n = seg_len == 64 ? 3 : 2;
  for (int k = 0; k < n; ++k)
    if ((uint32_t)set[k] >= col_rows - 1) return set[k];
  return 0;
}

template <bool XT, int TB>
static hl_status launch_stream_x(uint32_t seg_len, int jt, bool multi, dim3 grid, dim3 block, size_t lds,
                                 hipStream_t s, const StreamArgs& p) {
  if (seg_len == 64 && multi) {
    switch (jt) {
      case 12: return launch(gemv_stream_kernel<8, 12, XT, StreamArgs, false, TB>, grid, block, lds, s, p);
      case 16: return launch(gemv_stream_kernel<8, 16, XT, StreamArgs, false, TB>, grid, block, lds, s, p);
      case 20: return launch(gemv_stream_kernel<8, 20, XT, StreamArgs, false, TB>, grid, block, lds, s, p);
      default: return HL_EUNSUPPORTED;
    }
  }
  if (multi) return HL_EUNSUPPORTED;
  const GemvArgs& g = p.p;  // one matrix: the small argument block
  if (seg_len == 64) {
    switch (jt) {
      case 12: return launch(gemv_stream_kernel<8, 12, XT, GemvArgs, false, TB>, grid, block, lds, s, g);
      case 16: return launch(gemv_stream_kernel<8, 16, XT, GemvArgs, false, TB>, grid, block, lds, s, g);
      case 20: return launch(gemv_stream_kernel<8, 20, XT, GemvArgs, false, TB>, grid, block, lds, s, g);
      default: return HL_EUNSUPPORTED;
    }
  }
  if constexpr (TB == 0) {
    switch (jt) {
      case 8: return launch(gemv_stream_kernel<4, 8, XT, GemvArgs, false, 0>, grid, block, lds, s, g);
      case 12: return launch(gemv_stream_kernel<4, 12, XT, GemvArgs, false, 0>, grid, block, lds, s, g);
      default: return HL_EUNSUPPORTED;
    }
  }
  return HL_EUNSUPPORTED;
}

// The forms with NT = 2 or 4 tiles (17 to 32 or 33 to 64 activation rows):
// one matrix, x from its tiled copy (16 NT rows per 8-column chunk). Four
// tiles need columns of at least 16 words (their sums fill 4 KB of a wave's
// region).
static bool tiles_supported(int nt, uint32_t seg_len, int jt) {
  return nt == 2 || (nt == 4 && seg_len == 64 && jt >= 16);
}

template <int TB, int NT>
static hl_status launch_stream_tiles_tb(uint32_t seg_len, int jt, dim3 grid, dim3 block, size_t lds, hipStream_t s,
                                        const GemvArgs& g) {
  if (seg_len == 64) {
    switch (jt) {
      case 12:
        if constexpr (NT == 2)
          return launch(gemv_stream_kernel<8, 12, true, GemvArgs, false, TB, 2>, grid, block, lds, s, g);
        return HL_EUNSUPPORTED;
      case 16: return launch(gemv_stream_kernel<8, 16, true, GemvArgs, false, TB, NT>, grid, block, lds, s, g);
      case 20: return launch(gemv_stream_kernel<8, 20, true, GemvArgs, false, TB, NT>, grid, block, lds, s, g);
      default: return HL_EUNSUPPORTED;
    }
  }
  if constexpr (TB == 0 && NT == 2) {
    switch (jt) {
      case 8: return launch(gemv_stream_kernel<4, 8, true, GemvArgs, false, 0, 2>, grid, block, lds, s, g);
      case 12: return launch(gemv_stream_kernel<4, 12, true, GemvArgs, false, 0, 2>, grid, block, lds, s, g);
      default: return HL_EUNSUPPORTED;
    }
  }
  return HL_EUNSUPPORTED;
}

static hl_status launch_stream_tiles(int nt, bool bp, uint32_t seg_len, int jt, dim3 grid, dim3 block, size_t lds,
                                     hipStream_t s, const GemvArgs& g) {
  // eight waves: every tile's sums at the row-block end
  if (!tiles_supported(nt, seg_len, jt) || block.x != stream_threads(false, bp ? 1 : 0, nt)) return HL_EINVAL;
  if (nt == 4)
    return bp ? launch_stream_tiles_tb<1, 4>(seg_len, jt, grid, block, lds, s, g)
              : launch_stream_tiles_tb<0, 4>(seg_len, jt, grid, block, lds, s, g);
  return bp ? launch_stream_tiles_tb<1, 2>(seg_len, jt, grid, block, lds, s, g)
            : launch_stream_tiles_tb<0, 2>(seg_len, jt, grid, block, lds, s, g);
}

// Grouped launches (multi) exist for S = 64, bounded pairs (bp) for S = 64.
static hl_status launch_stream(bool xt, bool bp, uint32_t seg_len, int jt, bool multi, dim3 grid, dim3 block,
                               size_t lds, hipStream_t s, const StreamArgs& p) {
  // the bounded-pair table fill takes at most kBpPerThread entries per thread
  if (bp && block.x < kBpMinThreads) return HL_EINVAL;
  if (bp) return xt ? launch_stream_x<true, 1>(seg_len, jt, multi, grid, block, lds, s, p)
                    : launch_stream_x<false, 1>(seg_len, jt, multi, grid, block, lds, s, p);
  return xt ? launch_stream_x<true, 0>(seg_len, jt, multi, grid, block, lds, s, p)
            : launch_stream_x<false, 0>(seg_len, jt, multi, grid, block, lds, s, p);
}

// The float16 format on the persistent kernel (one matrix, float16 x; with
// DEC its decode to float16).
template <bool XT, bool DEC>
static hl_status launch_stream16_x(uint32_t seg_len, int jt, dim3 grid, dim3 block, size_t lds, hipStream_t s,
                                   const GemvArgs& g) {
  if (seg_len == 64) {
    switch (jt) {
      case 24: return launch(gemv_stream_kernel<8, 24, XT, GemvArgs, DEC, 2>, grid, block, lds, s, g);
      case 28: return launch(gemv_stream_kernel<8, 28, XT, GemvArgs, DEC, 2>, grid, block, lds, s, g);
      case 32: return launch(gemv_stream_kernel<8, 32, XT, GemvArgs, DEC, 2>, grid, block, lds, s, g);
      default: return HL_EUNSUPPORTED;
    }
  }
  switch (jt) {
    case 12: return launch(gemv_stream_kernel<4, 12, XT, GemvArgs, DEC, 2>, grid, block, lds, s, g);
    case 16: return launch(gemv_stream_kernel<4, 16, XT, GemvArgs, DEC, 2>, grid, block, lds, s, g);
    default: return HL_EUNSUPPORTED;
  }
}

static hl_status launch_stream16(bool xt, bool dec, uint32_t seg_len, int jt, dim3 grid, dim3 block, size_t lds,
                                 hipStream_t s, const GemvArgs& g) {
  if (dec) return launch_stream16_x<false, true>(seg_len, jt, grid, block, lds, s, g);
  return xt ? launch_stream16_x<true, false>(seg_len, jt, grid, block, lds, s, g)
            : launch_stream16_x<false, false>(seg_len, jt, grid, block, lds, s, g);
}

// Decoding to bf16 with the persistent kernel (p.y = the output).
static hl_status launch_stream_dec(uint32_t seg_len, int jt, bool bp, dim3 grid, dim3 block, size_t lds,
                                   hipStream_t s, const GemvArgs& p) {
  if (bp && block.x < kBpMinThreads) return HL_EINVAL;  // the bounded-pair table fill
  if (bp && seg_len == 64) {
    switch (jt) {
      case 12: return launch(gemv_stream_kernel<8, 12, false, GemvArgs, true, 1>, grid, block, lds, s, p);
      case 16: return launch(gemv_stream_kernel<8, 16, false, GemvArgs, true, 1>, grid, block, lds, s, p);
      case 20: return launch(gemv_stream_kernel<8, 20, false, GemvArgs, true, 1>, grid, block, lds, s, p);
      default: return HL_EUNSUPPORTED;
    }
  }
  if (seg_len == 64) {
    switch (jt) {
      case 12: return launch(gemv_stream_kernel<8, 12, false, GemvArgs, true, 0>, grid, block, lds, s, p);
      case 16: return launch(gemv_stream_kernel<8, 16, false, GemvArgs, true, 0>, grid, block, lds, s, p);
      case 20: return launch(gemv_stream_kernel<8, 20, false, GemvArgs, true, 0>, grid, block, lds, s, p);
      default: return HL_EUNSUPPORTED;
    }
  }
  switch (jt) {
    case 8: return launch(gemv_stream_kernel<4, 8, false, GemvArgs, true, 0>, grid, block, lds, s, p);
    case 12: return launch(gemv_stream_kernel<4, 12, false, GemvArgs, true, 0>, grid, block, lds, s, p);
    default: return HL_EUNSUPPORTED;
  }
}

// Segment lengths with a matrix-core instantiation (S = 8 * steps).
static bool mfma_steps_ok(uint32_t steps) {
  return steps == 1 || steps == 2 || steps == 4 || steps == 8 || steps == 16;
}

template <bool XT>
static hl_status launch_mfma_x(uint32_t steps, dim3 grid, dim3 block, size_t lds, hipStream_t s,
                               const GemvArgs& p) {
  switch (steps) {
    case 1: return launch(gemv_mfma_kernel<1, XT>, grid, block, lds, s, p);
    case 2: return launch(gemv_mfma_kernel<2, XT>, grid, block, lds, s, p);
    case 4: return launch(gemv_mfma_kernel<4, XT>, grid, block, lds, s, p);
    case 8: return launch(gemv_mfma_kernel<8, XT>, grid, block, lds, s, p);
    case 16: return launch(gemv_mfma_kernel<16, XT>, grid, block, lds, s, p);
    default: return HL_EUNSUPPORTED;
  }
}

static hl_status launch_mfma(bool xt, uint32_t steps, dim3 grid, dim3 block, size_t lds, hipStream_t s,
                             const GemvArgs& p) {
  return xt ? launch_mfma_x<true>(steps, grid, block, lds, s, p) : launch_mfma_x<false>(steps, grid, block, lds, s, p);
}

template <int B>
static hl_status launch_bf16_b(bool xbf16, dim3 grid, dim3 block, hipStream_t s, const uint16_t* w,
                               const void* x, float* y, uint32_t rows, uint32_t cols) {
  return xbf16 ? launch(gemv_bf16_kernel<B, true>, grid, block, 0, s, w, x, y, rows, cols)
               : launch(gemv_bf16_kernel<B, false>, grid, block, 0, s, w, x, y, rows, cols);
}

#define HL_BATCH_SWITCH(fn, batch, ...)                   \
  switch (batch) {                                        \
    case 1: return fn<1>(__VA_ARGS__);                    \
    case 2: return fn<2>(__VA_ARGS__);                    \
    case 3: return fn<3>(__VA_ARGS__);                    \
    case 4: return fn<4>(__VA_ARGS__);                    \
    case 5: return fn<5>(__VA_ARGS__);                    \
    case 6: return fn<6>(__VA_ARGS__);                    \
    case 7: return fn<7>(__VA_ARGS__);                    \
    case 8: return fn<8>(__VA_ARGS__);                    \
    case 9: return fn<9>(__VA_ARGS__);                    \
    case 10: return fn<10>(__VA_ARGS__);                  \
    case 11: return fn<11>(__VA_ARGS__);                  \
    case 12: return fn<12>(__VA_ARGS__);                  \
    case 13: return fn<13>(__VA_ARGS__);                  \
    case 14: return fn<14>(__VA_ARGS__);                  \
    case 15: return fn<15>(__VA_ARGS__);                  \
    case 16: return fn<16>(__VA_ARGS__);                  \
    default: return HL_EINVAL;                            \
  }

}  // namespace hl

using namespace hl;

// Buffers the kernels read or write in 16-byte pieces (activations, decoded
// weights, workspace, uncompressed weights) must be 16-byte aligned, fp32
// outputs 4-byte aligned; a null workspace is allowed where it is optional.
static bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

extern "C" hl_status hl_tensor_view(const void* blob_dev, const void* blob_host, size_t blob_bytes,
                                    uint32_t* lut_dev, hl_tensor* out) {
  if (!blob_dev || !blob_host || !lut_dev || !out || blob_bytes < HL_HEADER_BYTES) return HL_EINVAL;
  // the kernels copy the table and the group streams in 16-byte pieces
  if (!aligned(blob_dev, 16) || !aligned(lut_dev, 16)) return HL_EINVAL;
  Header H;
  uint32_t mseg = 0;
  const hl_status v = validate_blob(reinterpret_cast<const uint8_t*>(blob_host), blob_bytes, &H, &mseg);
  if (v != HL_OK) return v;
  hl_tensor t;
  std::memset(&t, 0, sizeof(t));
  t.blob_dev = reinterpret_cast<const uint8_t*>(blob_dev);
  t.lut_dev = lut_dev;
  t.rows = H.rows;
  t.cols = H.cols;
  t.n_seg = H.n_seg;
  t.n_grp = H.n_grp;
  t.total_bytes = H.total_bytes;
  t.off_seg_bits = H.off_seg_bits;
  t.off_grp_off = H.off_grp_off;
  t.off_stream = H.off_stream;
  t.off_raw = H.off_raw;
  t.seg_len = H.seg_len;
  t.grp_rows = H.grp_rows;
  t.lmax = H.lmax;
  t.max_grp_units = H.max_grp_units;
  t.max_seg_bits = mseg;
  t.format = H.format;
  t.cb = H.cb;
  t.cb8 = H.cb8;
  t.cb16 = H.cb16;
  *out = t;
  return HL_OK;
}

extern "C" hl_status hl_tensor_prepare(const hl_tensor* t, void* stream) {
  if (!t || !t->lut_dev) return HL_EINVAL;
  if (t->format == HL_FORMAT_FP16) {
    if (!code16_valid(t->cb16)) return HL_ECORRUPT;
    return launch(lut16_kernel, dim3(1), dim3(256), 0, (hipStream_t)stream, t->lut_dev, make_aux16(t->cb16),
                  tab16_layout(t->cb16));
  }
  if (t->format == HL_FORMAT_WHOLE_EXPONENT) {
    if (!code8_valid(t->cb8)) return HL_ECORRUPT;
    return launch(lut8_kernel, dim3(1), dim3(256), 0, (hipStream_t)stream, t->lut_dev, make_aux8(t->cb8));
  }
  if (t->format != HL_FORMAT_SPLIT) return HL_EINVAL;
  if (!field_code_valid(t->cb.eh, t->cb.lmax) || !field_code_valid(t->cb.el, t->cb.lmax)) return HL_ECORRUPT;
  Aux aux = make_aux(t->cb);
  return launch(lut_kernel, dim3(1), dim3(256), 0, (hipStream_t)stream, t->lut_dev, aux);
}


// Launch shape of the persistent kernel for one matrix: stream words per lane
// (*jt), waves per block (*waves) and LDS bytes per wave; false when the
// matrix does not fit it (16-row groups of the bf16 formats at S = 32 or 64,
// at least one row block per CU and two groups per wave of at least 8 waves
// per block, every segment within the largest stream word count).
// Longest code of a weight's exponent (the pair of the split format, the one
// code of the whole-exponent format), over the symbols present.
static uint32_t longest_exponent_code(const hl_tensor* t) {
  uint32_t a = 0, b = 0;
  if (t->format == HL_FORMAT_SPLIT) {
    for (int k = 0; k < 16; ++k) a = std::max<uint32_t>(a, t->cb.eh.len[k]), b = std::max<uint32_t>(b, t->cb.el.len[k]);
  } else if (t->format == HL_FORMAT_WHOLE_EXPONENT) {
    for (int k = 0; k < 256; ++k) a = std::max<uint32_t>(a, t->cb8.len[k]);
  } else {
    return 99;
  }
  return a + b;
}

// The persistent kernel's bounded-pair form applies (S = 64, pairs within
// the 11-bit window).
static bool bounded_pairs(const hl_tensor* t) {
  return t->seg_len == 64 && longest_exponent_code(t) <= (uint32_t)kBpBits;
}

static bool stream_shape(const hl_tensor* t, const GroupArgs& ga, int* jt, uint32_t* waves, size_t* per_wave) {
  if (t->grp_rows != 16 || (t->seg_len != 64 && t->seg_len != 32)) return false;
  const uint32_t CB = ga.CB, RB = ga.RB, cus = (uint32_t)device_cus();
  *jt = stream_rows_for(t->seg_len, ga.col_rows, is_fp16(t));
  const size_t tab = is_fp16(t)         ? (size_t)ga.t16_words * 4
                     : bounded_pairs(t) ? (size_t)kBpWords * 4
                                        : (size_t)(kLutN + kAuxWords) * 4;
  *per_wave = (size_t)(*jt + 1) * kCol * 4;
  uint32_t w = std::min<uint32_t>(kMaxWaves, stream_threads(false, is_fp16(t) ? 2 : 0) / 64);
  while (w > 1 && tab + w * *per_wave > kMaxLds) --w;
  // fewer waves per block when that gives every wave two groups: the
  // second group's loads then overlap the first one's decode
  while (w > 8 && (uint64_t)RB * CB < 2ull * cus * w) --w;
  *waves = w;
  // float16: two row blocks per CU at least (4096x4096, one per CU: 25.9 us
  // against 24.3 us on the non-persistent kernel; 14336x4096 65.8 against
  // 86.2 us)
  const uint32_t min_rb = is_fp16(t) ? 2 * cus : cus;
  return *jt && w >= 8 && CB >= w && RB >= min_rb && (uint64_t)RB * CB >= 2ull * cus * w;
}

extern "C" hl_status hl_decode(const hl_tensor* t, uint16_t* out_dev, void* stream) {
  if (!out_dev || !aligned(out_dev, 16)) return HL_EINVAL;
  Plan pl;
  hl_status st = make_plan(t, 0, !is_fp16(t), &pl);
  if (st != HL_OK) return st;
  const uint32_t n_grp = pl.ga.RB * pl.ga.CB;
  // large matrices: the persistent kernel, its product replaced by stores
  int jt = 0;
  uint32_t w = 0;
  size_t per_wave = 0;
  if (stream_shape(t, pl.ga, &jt, &w, &per_wave)) {
    GemvArgs p;
    std::memset(&p, 0, sizeof(p));
    p.g = pl.ga;
    p.y = reinterpret_cast<float*>(out_dev);
    p.B = 1;
    p.C = pl.ga.CB;
    p.KS = 1;
    // the kernel's bound when decoding (registers for a group's weights)
    w = stream_threads(true, is_fp16(t) ? 2 : 0) / 64;
    const dim3 grid(std::min<uint32_t>(pl.ga.RB, (uint32_t)device_cus()));
    // float16: its tables lead the dynamic LDS
    if (is_fp16(t))
      return launch_stream16(false, true, t->seg_len, jt, grid, dim3(w * 64),
                             (size_t)pl.ga.t16_words * 4 + w * per_wave, (hipStream_t)stream, p);
    // the bounded-pair table where the encoder's joint limit holds (with the
    // whole-row stores it decodes 28672x8192 in 175.9 us against 187.7 us
    // with the joint table; stored straight from the lanes, 307 against 273)
    return launch_stream_dec(t->seg_len, jt, bounded_pairs(t),
                             dim3(std::min<uint32_t>(pl.ga.RB, (uint32_t)device_cus())), dim3(w * 64), w * per_wave,
                             (hipStream_t)stream, p);
  }
  if (is_fp16(t)) {
    const uint32_t per_cu = std::max<uint32_t>(1, std::min<uint32_t>(8, kMaxLds / (uint32_t)pl.lds));
    const uint32_t blocks = std::min<uint32_t>((n_grp + pl.waves - 1) / pl.waves, device_cus() * per_cu);
    return launch(decode16_kernel, dim3(blocks), dim3(pl.waves * 64), pl.lds, (hipStream_t)stream, pl.ga,
                  out_dev);
  }
  const uint32_t per_cu =
      std::max<uint32_t>(1, std::min<uint32_t>(8, kMaxLds / (uint32_t)(pl.lds + (kLutN + kAuxWords) * 4)));
  const uint32_t blocks = std::min<uint32_t>((n_grp + pl.waves - 1) / pl.waves, device_cus() * per_cu);
  return launch(decode_kernel, dim3(blocks), dim3(pl.waves * 64), pl.lds, (hipStream_t)stream, pl.ga,
                out_dev);
}

static uint32_t ks_cap(uint32_t CB) { return std::min<uint32_t>(CB, 64); }

// Workspace layout: the tiled copy of bf16 activations (batch above one,
// 16-row groups: 32 bytes per column), then RB arrival counters and the
// split partial sums of the non-persistent kernels.
static uint64_t xtile_region(const hl_tensor* t, uint32_t batch) {
  return (batch > 1 && t->grp_rows == 16) ? ((uint64_t)t->cols * 32 + 255) & ~255ull : 0;
}
static uint64_t counter_bytes(uint32_t RB) { return ((uint64_t)RB * 4 + 255) & ~255ull; }

// Column blocks per block (*C) and blocks per row block (*KS) of the
// non-persistent kernels: enough blocks to fill the device, each wave
// decoding at least one group.
static void split_shape(const Plan& pl, uint32_t* C_out, uint32_t* KS_out) {
  const uint32_t CB = pl.ga.CB, RB = pl.ga.RB;
  const uint32_t cus = (uint32_t)device_cus();
  const uint64_t target_waves = (uint64_t)cus * 16;
  const uint32_t gpw = (uint32_t)std::max<uint64_t>(1, ((uint64_t)RB * CB + target_waves - 1) / target_waves);
  uint32_t C = std::min<uint32_t>(CB, pl.waves * gpw);
  uint32_t KS = (CB + C - 1) / C;
  // a matrix with fewer row blocks than CUs: split its columns further, so
  // that every CU gets a block (narrower blocks, one group per wave)
  if ((uint64_t)RB * KS < cus) {
    KS = std::min<uint32_t>(CB, (cus + RB - 1) / RB);
    C = (CB + KS - 1) / KS;
    KS = (CB + C - 1) / C;
  }
  if (KS > ks_cap(CB)) {
    KS = ks_cap(CB);
    C = (CB + KS - 1) / KS;
    KS = (CB + C - 1) / C;
  }
  *C_out = C;
  *KS_out = KS;
}

// Workspace bytes of a split over KS k-parts (counters and partial sums).
static uint64_t split_bytes(const Plan& pl, uint32_t batch, uint32_t KS) {
  return KS > 1 ? counter_bytes(pl.ga.RB) + (uint64_t)KS * batch * pl.ga.RB * pl.ga.GR * 4 : 0;
}

__global__ void __launch_bounds__(256) zero_kernel(uint32_t* p, uint32_t n) {
  for (uint32_t k = blockIdx.x * blockDim.x + threadIdx.x; k < n; k += gridDim.x * blockDim.x) p[k] = 0;
}

// Split of the non-persistent kernels, with room for partials in the
// workspace (else one block per row block). *block_waves = the waves a block
// is launched with (no more than its column blocks). With `clear`, the
// arrival counters are zeroed by a small kernel on `stream` first (a
// workspace shared with calls of other shapes, whose bytes there are not
// counters).
static hl_status choose_split(const hl_tensor* t, const Plan& pl, uint32_t batch, void* workspace_dev,
                              size_t workspace_bytes, bool clear, hipStream_t stream, GemvArgs* p,
                              uint32_t* block_waves) {
  uint32_t C = 0, KS = 0;
  split_shape(pl, &C, &KS);
  const uint64_t base = xtile_region(t, batch);
  if (KS > 1 && (!workspace_dev || workspace_bytes < base + split_bytes(pl, batch, KS))) {
    KS = 1;  // no room for partial sums: one block per row block
    C = pl.ga.CB;
  }
  p->C = C;
  p->KS = KS;
  *block_waves = std::min<uint32_t>(pl.waves, C);
  if (KS > 1) {
    uint8_t* w = reinterpret_cast<uint8_t*>(workspace_dev) + base;
    p->counter = reinterpret_cast<uint32_t*>(w);
    p->partial = reinterpret_cast<float*>(w + counter_bytes(pl.ga.RB));
    if (clear) return launch(zero_kernel, dim3((pl.ga.RB + 255) / 256), dim3(256), 0, stream, p->counter, pl.ga.RB);
  }
  return HL_OK;
}

template <bool XT>
static hl_status launch_mfma16_x(uint32_t steps, dim3 grid, dim3 block, size_t lds, hipStream_t s,
                                 const GemvArgs& p) {
  switch (steps) {
    case 1: return launch(gemv16_mfma_kernel<1, XT>, grid, block, lds, s, p);
    case 2: return launch(gemv16_mfma_kernel<2, XT>, grid, block, lds, s, p);
    case 4: return launch(gemv16_mfma_kernel<4, XT>, grid, block, lds, s, p);
    case 8: return launch(gemv16_mfma_kernel<8, XT>, grid, block, lds, s, p);
    case 16: return launch(gemv16_mfma_kernel<16, XT>, grid, block, lds, s, p);
    default: return HL_EUNSUPPORTED;
  }
}

static hl_status launch_mfma16(bool xt, uint32_t steps, dim3 grid, dim3 block, size_t lds, hipStream_t s,
                               const GemvArgs& p) {
  return xt ? launch_mfma16_x<true>(steps, grid, block, lds, s, p)
            : launch_mfma16_x<false>(steps, grid, block, lds, s, p);
}

// Larger batches on the matrix cores read the activations from a tiled copy
// in the workspace (when it is large enough): the copy costs a launch (about
// 2.5 us), and reading 16 rows per 8-column chunk costs more the larger the
// batch and the matrix (4096x4096: +1.5 us at batch 8; 28672x8192: +3.5 us at
// batch 4, +41 us at batch 8, +109 us at batch 16; the 8B layer's grouped
// step at batch 5-7 124-142 us read directly, 120 us tiled at batch 8). On
// success with a tiled copy, p->x points to it and *xt is set.
static hl_status tile_activations(const hl_tensor* t, const void* x_dev, uint32_t batch, void* workspace_dev,
                                  size_t workspace_bytes, hipStream_t stream, GemvArgs* p, bool* xt) {
  *xt = false;
  const uint64_t n = t->rows * t->cols;
  const bool want = batch >= 12 || (batch >= 5 && n >= (32ull << 20)) || (batch >= 4 && n >= (128ull << 20));
  if (!want || !workspace_dev || workspace_bytes < xtile_region(t, batch)) return HL_OK;
  uint4* tile = reinterpret_cast<uint4*>(workspace_dev);
  const uint32_t chunks = (uint32_t)(t->cols / 8);
  const hl_status st = launch(xtile_kernel<16>, dim3((chunks * 16 + 255) / 256), dim3(256), 0, stream,
                              reinterpret_cast<const uint4*>(x_dev), batch, chunks, tile);
  if (st != HL_OK) return st;
  p->x = tile;
  *xt = true;
  return HL_OK;
}

// Float16 format (16-row groups, float16 x): the persistent kernel's float16
// form for large matrices, else the matrix-core kernel.
static hl_status gemv16(const hl_tensor* t, const void* x_dev, uint32_t batch, float* y_dev, void* workspace_dev,
                        size_t workspace_bytes, bool clear, hipStream_t stream) {
  if (t->grp_rows != 16 || t->seg_len % 8 || !mfma_steps_ok(t->seg_len / 8)) return HL_EUNSUPPORTED;
  Plan pl;
  hl_status st = make_plan(t, 0, false, &pl);
  if (st != HL_OK) return st;
  GemvArgs p;
  std::memset(&p, 0, sizeof(p));
  p.g = pl.ga;
  p.x = x_dev;
  p.y = y_dev;
  p.B = batch;
  // large matrices: the persistent kernel (S = 32 or 64, a row block per CU
  // and two groups per wave), its tables ahead of the wave regions
  int jt = 0;
  uint32_t w = 0;
  size_t per_wave = 0;
  bool xt = false;
  if (stream_shape(t, pl.ga, &jt, &w, &per_wave)) {
    st = tile_activations(t, x_dev, batch, workspace_dev, workspace_bytes, stream, &p, &xt);
    if (st != HL_OK) return st;
    p.C = pl.ga.CB;
    p.KS = 1;
    return launch_stream16(xt, false, t->seg_len, jt, dim3(std::min<uint32_t>(pl.ga.RB, (uint32_t)device_cus())),
                           dim3(w * 64), (size_t)pl.ga.t16_words * 4 + w * per_wave, stream, p);
  }
  st = choose_split(t, pl, batch, workspace_dev, workspace_bytes, clear, stream, &p, &w);
  if (st != HL_OK) return st;
  st = tile_activations(t, x_dev, batch, workspace_dev, workspace_bytes, stream, &p, &xt);
  if (st != HL_OK) return st;
  const dim3 grid(pl.ga.RB * p.KS), block(w * 64);
  // the reduction reuses the wave regions: 4 floats per lane per wave
  const size_t lds = std::max<size_t>(pl.lds_for(w), (size_t)pl.ga.t16_words * 4 + (size_t)w * 4 * 64 * 4);
  return launch_mfma16(xt, t->seg_len / 8, grid, block, lds, stream, p);
}

// Which kernel family a product runs on and its plan: 16-row groups with
// bf16 activations run on the matrix cores (the persistent kernel where it
// fits, *persistent); the vector kernel stages raw bytes and the activation
// slice (GC*S columns per batch row, *x_words) in LDS.
static hl_status gemv_plan(const hl_tensor* t, hl_dtype x_dtype, uint32_t batch, Plan* pl, bool* mfma,
                           bool* persistent, uint32_t* x_words) {
  const bool xb = x_dtype == HL_BF16;
  *mfma = xb && t->grp_rows == 16 && t->seg_len % 8 == 0 && mfma_steps_ok(t->seg_len / 8);
  const uint32_t slice = (HL_GROUP_SEGS / t->grp_rows) * t->seg_len;
  *x_words = xb ? slice * batch / 2 : slice * batch;
  const hl_status st = make_plan(t, *mfma ? 0 : *x_words, !*mfma, pl);
  if (st != HL_OK) return st;
  int jt = 0;
  uint32_t w = 0;
  size_t per_wave = 0;
  *persistent = *mfma && stream_shape(t, pl->ga, &jt, &w, &per_wave);
  return HL_OK;
}

// Workspace bytes a product uses at most (tiled activations, counters and
// partial sums); 0 for bad arguments.
static uint64_t gemv_need(const hl_tensor* t, hl_dtype x_dtype, uint32_t batch) {
  Plan pl;
  if (is_fp16(t)) {
    if (x_dtype != HL_F16 || make_plan(t, 0, false, &pl) != HL_OK) return 0;
    int jt = 0;
    uint32_t w = 0;
    size_t per_wave = 0;
    if (stream_shape(t, pl.ga, &jt, &w, &per_wave)) return xtile_region(t, batch);
  } else {
    bool mfma = false, persistent = false;
    uint32_t xw = 0;
    if (x_dtype == HL_F16 || gemv_plan(t, x_dtype, batch, &pl, &mfma, &persistent, &xw) != HL_OK) return 0;
    if (persistent) return xtile_region(t, batch);
  }
  uint32_t C = 0, KS = 0;
  split_shape(pl, &C, &KS);
  return xtile_region(t, batch) + split_bytes(pl, batch, KS);
}

extern "C" size_t hl_gemv_workspace_bytes(const hl_tensor* t, uint32_t batch) {
  if (!t || t->seg_len == 0 || t->grp_rows == 0 || t->grp_rows > HL_GROUP_SEGS || batch < 1 ||
      batch > HL_MAX_BATCH)
    return 0;
  if (is_fp16(t)) return (size_t)gemv_need(t, HL_F16, batch);
  return (size_t)std::max(gemv_need(t, HL_F32, batch), gemv_need(t, HL_BF16, batch));
}

static hl_status gemv_args_ok(const hl_tensor* t, const void* x_dev, hl_dtype x_dtype, uint32_t batch,
                              const float* y_dev) {
  if (!t || !x_dev || !y_dev || batch < 1 || batch > HL_MAX_BATCH ||
      (x_dtype != HL_F32 && x_dtype != HL_BF16 && x_dtype != HL_F16))
    return HL_EINVAL;
  if (!aligned(x_dev, 16) || !aligned(y_dev, 4)) return HL_EINVAL;
  if (t->grp_rows == 0 || t->grp_rows > HL_GROUP_SEGS || t->seg_len == 0) return HL_EINVAL;
  if (is_fp16(t) != (x_dtype == HL_F16)) return HL_EUNSUPPORTED;
  return HL_OK;
}

// The product of hl_decode_gemv; `clear`: zero the split's arrival counters
// first (the workspace may hold other bytes there).
static hl_status gemv_impl(const hl_tensor* t, const void* x_dev, hl_dtype x_dtype, uint32_t batch, float* y_dev,
                           void* workspace_dev, size_t workspace_bytes, bool clear, hipStream_t stream) {
  if (is_fp16(t)) return gemv16(t, x_dev, batch, y_dev, workspace_dev, workspace_bytes, clear, stream);
  Plan pl;
  bool mfma = false, persistent = false;
  uint32_t x_words = 0;
  hl_status st = gemv_plan(t, x_dtype, batch, &pl, &mfma, &persistent, &x_words);
  if (st != HL_OK) return st;
  const bool xb = x_dtype == HL_BF16;
  GemvArgs p;
  std::memset(&p, 0, sizeof(p));
  p.g = pl.ga;
  p.x = x_dev;
  p.y = y_dev;
  p.x_words = mfma ? 0 : x_words;
  p.B = batch;
  const uint32_t CB = pl.ga.CB, RB = pl.ga.RB;
  const uint32_t cus = (uint32_t)device_cus();
  bool xt = false;
  if (mfma) {
    st = tile_activations(t, x_dev, batch, workspace_dev, workspace_bytes, stream, &p, &xt);
    if (st != HL_OK) return st;
  }
  // Persistent kernel: S = 32 or 64, at least one row block per CU and two
  // groups per wave.
  if (persistent) {
    int jt = 0;
    uint32_t w = 0;
    size_t per_wave = 0;
    if (stream_shape(t, pl.ga, &jt, &w, &per_wave)) {
      p.C = CB;
      p.KS = 1;
      StreamArgs sa;  // one matrix: only sa.p (with p.g, p.y) reaches the kernel
      std::memset(&sa, 0, sizeof(sa));
      sa.p = p;
      sa.n = 1;
      sa.part0[1] = std::min(RB, cus);
      const bool bp = bounded_pairs(t);
      return launch_stream(xt, bp, t->seg_len, jt, false, dim3(sa.part0[1]), dim3(w * 64), w * per_wave,
                           stream, sa);
    }
  }
  // Column blocks per block and blocks per row block.
  uint32_t w = 0;
  st = choose_split(t, pl, batch, workspace_dev, workspace_bytes, clear, stream, &p, &w);
  if (st != HL_OK) return st;
  const uint32_t KS = p.KS;
  const dim3 grid(RB * KS), block(w * 64);
  if (mfma) {
    // the reduction reuses the wave regions: 4 floats per lane per wave
    const size_t lds = std::max<size_t>(pl.lds_for(w), (size_t)w * 4 * 64 * 4);
    return launch_mfma(xt, t->seg_len / 8, grid, block, lds, stream, p);
  }
  const size_t lds = std::max<size_t>(pl.lds_for(w), (size_t)w * batch * 64 * 4);
  HL_BATCH_SWITCH(launch_gemv_b, batch, xb, grid, block, lds, stream, p);
}

extern "C" hl_status hl_decode_gemv(const hl_tensor* t, const void* x_dev, hl_dtype x_dtype, uint32_t batch,
                                    float* y_dev, void* workspace_dev, size_t workspace_bytes, void* stream) {
  const hl_status st = gemv_args_ok(t, x_dev, x_dtype, batch, y_dev);
  if (st != HL_OK) return st;
  if (!aligned(workspace_dev, 16)) return HL_EINVAL;
  return gemv_impl(t, x_dev, x_dtype, batch, y_dev, workspace_dev, workspace_bytes, false, (hipStream_t)stream);
}

// ------------------------------------------------------------------ allocation-free product

// Scratch memory of hl_decode_gemv_noalloc: one array per GPU the library
// runs on, held until the process ends. In host code `scratch` is a
// stand-in, not a device address: the address of a GPU's copy comes from
// hipGetSymbolAddress (with that GPU current) and is what the kernels get.
static __device__ __align__(256) uint8_t scratch[HL_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch[kMaxDevices];

// The current GPU's scratch address, looked up once per GPU.
static hl_status scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return HL_EHIP;
  if (dev >= kMaxDevices) return HL_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return HL_EHIP;
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return HL_OK;
}

extern "C" hl_status hl_decode_gemv_noalloc(const hl_tensor* t, const void* x_dev, hl_dtype x_dtype, uint32_t batch,
                                            float* y_dev, void* stream) {
  hl_status st = gemv_args_ok(t, x_dev, x_dtype, batch, y_dev);
  if (st != HL_OK) return st;
  const uint64_t need = gemv_need(t, x_dtype, batch);
  if (need > HL_NOALLOC_SCRATCH_BYTES) return HL_EUNSUPPORTED;
  void* ws = nullptr;
  st = scratch_address(&ws);
  if (st != HL_OK) return st;
  return gemv_impl(t, x_dev, x_dtype, batch, y_dev, ws, HL_NOALLOC_SCRATCH_BYTES, true, (hipStream_t)stream);
}

// Shape of a grouped launch of the persistent kernel over ts[0..count) (bf16
// formats, 16-row groups, S = 64, bf16 x): the plans, stream words per lane,
// waves per block, the bounded-pair form, and the blocks per matrix (one
// each, then one more at a time to the matrix with the most row blocks per
// block, until every CU has a block). False when the matrices do not take it.
struct GroupShape {
  Plan pl[kMaxParts];
  int jt;
  uint32_t w, nb[kMaxParts], used;
  bool bp;
  size_t per_wave;
};

static bool group_shape(const hl_tensor* const* ts, uint32_t count, GroupShape* g) {
  if (count < 2 || count > kMaxParts) return false;
  for (uint32_t k = 0; k < count; ++k)
    if (!ts[k] || is_fp16(ts[k]) || ts[k]->grp_rows != 16 || ts[k]->seg_len != 64 || ts[k]->cols != ts[0]->cols)
      return false;
  const uint32_t cus = (uint32_t)device_cus();
  g->jt = 0;
  uint64_t groups = 0, rbs = 0;
  for (uint32_t k = 0; k < count; ++k) {
    if (make_plan(ts[k], 0, false, &g->pl[k]) != HL_OK) return false;
    const int j = stream_rows_for(ts[k]->seg_len, g->pl[k].ga.col_rows, false);
    if (j == 0) return false;
    g->jt = std::max(g->jt, j);
    groups += (uint64_t)g->pl[k].ga.RB * g->pl[k].ga.CB;
    rbs += g->pl[k].ga.RB;
  }
  g->bp = true;  // the bounded-pair kernel when every matrix has bounded pairs
  for (uint32_t k = 0; k < count && g->bp; ++k) g->bp = bounded_pairs(ts[k]);
  const size_t tab = g->bp ? (size_t)kBpWords * 4 : (size_t)(kLutN + kAuxWords) * 4;
  g->per_wave = (size_t)(g->jt + 1) * kCol * 4;
  uint32_t w = kMaxWaves;
  while (w > 1 && tab + w * g->per_wave > kMaxLds) --w;
  while (w > 8 && groups < 2ull * cus * w) --w;
  if (!(w >= 8 && g->pl[0].ga.CB >= w && rbs >= cus)) return false;
  g->w = w;
  g->used = count;
  for (uint32_t k = 0; k < count; ++k) g->nb[k] = 1;
  while (g->used < cus) {
    uint32_t best = 0, worst = 0;
    for (uint32_t k = 0; k < count; ++k) {
      const uint32_t per = (g->pl[k].ga.RB + g->nb[k] - 1) / g->nb[k];
      if (per > worst || (per == worst && g->pl[k].ga.RB > g->pl[best].ga.RB)) worst = per, best = k;
    }
    if (worst <= 1) break;
    ++g->nb[best];
    ++g->used;
  }
  return true;
}

static hl_status gemv_multi_impl(const hl_tensor* const* ts, uint32_t count, const void* x_dev, hl_dtype x_dtype,
                                 uint32_t batch, float* const* y_devs, void* workspace_dev, size_t workspace_bytes,
                                 hipStream_t stream) {
  if (!ts || !y_devs || !x_dev || count < 1 || count > kMaxParts || batch < 1 || batch > HL_MAX_BATCH)
    return HL_EINVAL;
  if (!aligned(x_dev, 16) || !aligned(workspace_dev, 16)) return HL_EINVAL;
  for (uint32_t k = 0; k < count; ++k)
    if (!ts[k] || !y_devs[k] || !aligned(y_devs[k], 4) || ts[k]->cols != ts[0]->cols) return HL_EINVAL;
  // One launch of the persistent kernel when every matrix has its container
  // geometry (bf16 formats, 16-row groups, S = 64) and bf16 x; otherwise the
  // matrices one after another.
  GroupShape g;
  if (!(x_dtype == HL_BF16 && group_shape(ts, count, &g))) {
    // one product after another on the shared workspace: a split product
    // zeroes its counters first (another matrix's product may have left
    // partial sums where they lie)
    for (uint32_t k = 0; k < count; ++k) {
      hl_status st = gemv_args_ok(ts[k], x_dev, x_dtype, batch, y_devs[k]);
      if (st == HL_OK)
        st = gemv_impl(ts[k], x_dev, x_dtype, batch, y_devs[k], workspace_dev, workspace_bytes, count > 1, stream);
      if (st != HL_OK) return st;
    }
    return HL_OK;
  }
  GemvArgs p;
  std::memset(&p, 0, sizeof(p));
  p.x = x_dev;
  p.B = batch;
  p.C = g.pl[0].ga.CB;
  p.KS = 1;
  bool xt = false;
  uint32_t big = 0;  // the tiled activations go where the largest matrix's workspace puts them
  for (uint32_t k = 1; k < count; ++k) big = ts[k]->rows > ts[big]->rows ? k : big;
  const hl_status st = tile_activations(ts[big], x_dev, batch, workspace_dev, workspace_bytes, stream, &p, &xt);
  if (st != HL_OK) return st;
  StreamArgs sa;
  std::memset(&sa, 0, sizeof(sa));
  sa.p = p;
  sa.n = count;
  for (uint32_t k = 0; k < count; ++k) {
    sa.g[k] = g.pl[k].ga;
    sa.y[k] = y_devs[k];
    sa.part0[k + 1] = sa.part0[k] + g.nb[k];
  }
  return launch_stream(xt, g.bp, ts[0]->seg_len, g.jt, true, dim3(g.used), dim3(g.w * 64), g.w * g.per_wave,
                       stream, sa);
}

extern "C" hl_status hl_decode_gemv_multi(const hl_tensor* const* ts, uint32_t count, const void* x_dev,
                                          hl_dtype x_dtype, uint32_t batch, float* const* y_devs,
                                          void* workspace_dev, size_t workspace_bytes, void* stream) {
  return gemv_multi_impl(ts, count, x_dev, x_dtype, batch, y_devs, workspace_dev, workspace_bytes,
                         (hipStream_t)stream);
}

// ------------------------------------------------------------------ prefill GEMM host side

constexpr uint32_t kGemmMaxTiles = 8;  // token tiles of 16 per block

static uint32_t gemm_row_sets(const hl_tensor* t) { return (uint32_t)((t->rows + 255) / 256); }

// Prefill above this many tokens: the weights are decoded once to bf16 in the
// workspace and multiplied by the vendor GEMM (hipBLASLt). Up to it the
// persistent kernel's tiled forms, or the fused kernel that decodes each tile
// once per chunk of tokens (4096x4096, cold: decode + GEMM 32.9-36.9 us at 65
// to 112 tokens against 42.6-48.2 us fused; 39.3 us at 128, 45.4 us at 512).
constexpr uint32_t kGemmFusedMaxTokens = 64;
constexpr uint32_t kTile = 16;  // activation rows of one matrix-instruction tile

extern "C" size_t hl_gemm_workspace_bytes(const hl_tensor* t, uint32_t tokens) {
  if (!t || tokens == 0 || t->seg_len == 0 || t->grp_rows != 16) return 0;
  if (tokens > kGemmFusedMaxTokens) return (size_t)(t->rows * t->cols * 2);  // the decoded weights
  const uint64_t CB = (t->cols / t->seg_len) / 4;
  return (size_t)(CB * tokens * t->rows * 4);
}

// One hipBLASLt handle per GPU, created on first use with that GPU current.
static std::mutex g_lt_mu;
static hipblasLtHandle_t g_lt[kMaxDevices];

static hl_status lt_handle(hipblasLtHandle_t* out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return HL_EHIP;
  if (dev >= kMaxDevices) return HL_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_lt_mu);
  if (!g_lt[dev] && hipblasLtCreate(&g_lt[dev]) != HIPBLAS_STATUS_SUCCESS) {
    g_lt[dev] = nullptr;
    return HL_EHIP;
  }
  *out = g_lt[dev];
  return HL_OK;
}

// Y[n][r] = sum_k W[r][k] X[n][k] from bf16 W [rows][cols] and X [tokens][cols]
// into float32 Y [tokens][rows]: in column-major terms D (rows x tokens, ld
// rows) = A^T B with A = W as a cols x rows matrix and B = X as cols x tokens.
// No GEMM workspace (an algorithm that needs none), so nothing is cleared on
// the stream.
static hl_status gemm_bf16_lt(const uint16_t* w, const uint16_t* x, float* y, uint64_t rows, uint64_t cols,
                              uint32_t tokens, hipStream_t stream) {
  hipblasLtHandle_t h = nullptr;
  hl_status st = lt_handle(&h);
  if (st != HL_OK) return st;
  hipblasLtMatmulDesc_t op = nullptr;
  hipblasLtMatrixLayout_t la = nullptr, lb = nullptr, ld = nullptr;
  hipblasLtMatmulPreference_t pref = nullptr;
  st = HL_EHIP;
  const hipblasOperation_t ta = HIPBLAS_OP_T, tb = HIPBLAS_OP_N;
  const uint64_t no_ws = 0;
  hipblasLtMatmulHeuristicResult_t heur[1];
  int found = 0;
  const float alpha = 1.f, beta = 0.f;
  if (hipblasLtMatmulDescCreate(&op, HIPBLAS_COMPUTE_32F, HIP_R_32F) == HIPBLAS_STATUS_SUCCESS &&
      hipblasLtMatmulDescSetAttribute(op, HIPBLASLT_MATMUL_DESC_TRANSA, &ta, sizeof(ta)) == HIPBLAS_STATUS_SUCCESS &&
      hipblasLtMatmulDescSetAttribute(op, HIPBLASLT_MATMUL_DESC_TRANSB, &tb, sizeof(tb)) == HIPBLAS_STATUS_SUCCESS &&
      hipblasLtMatrixLayoutCreate(&la, HIP_R_16BF, cols, rows, (int64_t)cols) == HIPBLAS_STATUS_SUCCESS &&
      hipblasLtMatrixLayoutCreate(&lb, HIP_R_16BF, cols, tokens, (int64_t)cols) == HIPBLAS_STATUS_SUCCESS &&
      hipblasLtMatrixLayoutCreate(&ld, HIP_R_32F, rows, tokens, (int64_t)rows) == HIPBLAS_STATUS_SUCCESS &&
      hipblasLtMatmulPreferenceCreate(&pref) == HIPBLAS_STATUS_SUCCESS &&
      hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &no_ws,
                                            sizeof(no_ws)) == HIPBLAS_STATUS_SUCCESS) {
    if (hipblasLtMatmulAlgoGetHeuristic(h, op, la, lb, ld, ld, pref, 1, heur, &found) != HIPBLAS_STATUS_SUCCESS ||
        found < 1)
      st = HL_EUNSUPPORTED;
    else if (hipblasLtMatmul(h, op, &alpha, w, la, x, lb, &beta, y, ld, y, ld, &heur[0].algo, nullptr, 0,
                             stream) == HIPBLAS_STATUS_SUCCESS)
      st = HL_OK;
  }
  if (pref) hipblasLtMatmulPreferenceDestroy(pref);
  if (ld) hipblasLtMatrixLayoutDestroy(ld);
  if (lb) hipblasLtMatrixLayoutDestroy(lb);
  if (la) hipblasLtMatrixLayoutDestroy(la);
  if (op) hipblasLtMatmulDescDestroy(op);
  return st;
}

template <int SP>
static hl_status launch_gemm_sp(uint32_t nt, dim3 grid, size_t lds, hipStream_t s, const GemmArgs& p) {
  switch (nt) {
    case 1: return launch(gemm_mfma_kernel<SP, 1>, grid, dim3(1024), lds, s, p);
    case 2: return launch(gemm_mfma_kernel<SP, 2>, grid, dim3(1024), lds, s, p);
    case 4: return launch(gemm_mfma_kernel<SP, 4>, grid, dim3(1024), lds, s, p);
    case 8: return launch(gemm_mfma_kernel<SP, 8>, grid, dim3(1024), lds, s, p);
    default: return HL_EUNSUPPORTED;
  }
}

extern "C" hl_status hl_decode_gemm(const hl_tensor* t, const void* x_dev, hl_dtype x_dtype, uint32_t tokens,
                                    float* y_dev, void* workspace_dev, size_t workspace_bytes, void* stream) {
  if (!t || !x_dev || !y_dev || tokens == 0 || tokens >= (1u << 24)) return HL_EINVAL;
  if (!aligned(x_dev, 16) || !aligned(y_dev, 4) || !aligned(workspace_dev, 16)) return HL_EINVAL;
  if (x_dtype != HL_BF16 || is_fp16(t) || t->grp_rows != 16 || (t->seg_len != 32 && t->seg_len != 64))
    return HL_EUNSUPPORTED;
  if (!workspace_dev || workspace_bytes < hl_gemm_workspace_bytes(t, tokens)) return HL_EINVAL;
  if (tokens <= 4 * kTile) {
    // up to 64 tokens on matrices the persistent kernel takes: one, two or
    // four 16-token tiles per step of its decode, each row block summed in
    // its block (no partial sums); the activations tiled in the workspace (16
    // rows per tile and 8-column chunk, so that a wave's reads of one chunk
    // are contiguous)
    Plan pp;
    hl_status sp = make_plan(t, 0, false, &pp);
    if (sp != HL_OK) return sp;
    int jt = 0;
    uint32_t w = 0;
    size_t per_wave = 0;
    const int nt = tokens <= kTile ? 1 : tokens <= 2 * kTile ? 2 : 4;
    if (stream_shape(t, pp.ga, &jt, &w, &per_wave) && (nt == 1 || tiles_supported(nt, t->seg_len, jt))) {
      GemvArgs p;
      std::memset(&p, 0, sizeof(p));
      p.g = pp.ga;
      p.x = x_dev;
      p.y = y_dev;
      p.B = tokens;
      p.C = pp.ga.CB;
      p.KS = 1;
      const bool bp = bounded_pairs(t);
      const dim3 grid(std::min<uint32_t>(pp.ga.RB, (uint32_t)device_cus()));
      if (nt > 1) {
        const uint32_t chunks = (uint32_t)(t->cols / 8), R = nt * kTile;
        if (workspace_bytes < (size_t)chunks * R * 16) return HL_EINVAL;
        uint4* tile = reinterpret_cast<uint4*>(workspace_dev);
        const dim3 tgrid((chunks * R + 255) / 256);
        const uint4* xs = reinterpret_cast<const uint4*>(x_dev);
        sp = nt == 2 ? launch(xtile_kernel<2 * kTile>, tgrid, dim3(256), 0, (hipStream_t)stream, xs, tokens, chunks, tile)
                     : launch(xtile_kernel<4 * kTile>, tgrid, dim3(256), 0, (hipStream_t)stream, xs, tokens, chunks, tile);
        if (sp != HL_OK) return sp;
        p.x = tile;
        w = stream_threads(false, bp ? 1 : 0, nt) / 64;
        return launch_stream_tiles(nt, bp, t->seg_len, jt, grid, dim3(w * 64), w * per_wave, (hipStream_t)stream, p);
      }
      bool xt = false;
      sp = tile_activations(t, x_dev, tokens, workspace_dev, workspace_bytes, (hipStream_t)stream, &p, &xt);
      if (sp != HL_OK) return sp;
      StreamArgs sa;
      std::memset(&sa, 0, sizeof(sa));
      sa.p = p;
      sa.n = 1;
      sa.part0[1] = grid.x;
      return launch_stream(xt, bp, t->seg_len, jt, false, grid, dim3(w * 64), w * per_wave,
                           (hipStream_t)stream, sa);
    }
  }
  if (tokens > kGemmFusedMaxTokens) {
    // many tokens: decode once (bit-exact bf16 in the workspace), then the GEMM
    uint16_t* w = reinterpret_cast<uint16_t*>(workspace_dev);
    const hl_status st = hl_decode(t, w, stream);
    if (st != HL_OK) return st;
    return gemm_bf16_lt(w, reinterpret_cast<const uint16_t*>(x_dev), y_dev, t->rows, t->cols, tokens,
                        (hipStream_t)stream);
  }
  Plan pl;
  hl_status st = make_plan(t, 0, false, &pl);
  if (st != HL_OK) return st;
  const uint32_t SP = t->seg_len / 8;
  // Token tiles per block: as many as the tokens need (a power of two, at
  // most 8) and the LDS holds next to 16 waves' stream columns and the table.
  const size_t cols_bytes = (size_t)16 * pl.ga.col_rows * kCol * 4;
  const size_t tab = (size_t)(kLutN + kAuxWords) * 4;
  uint32_t nt = 1;
  while (nt < kGemmMaxTiles && nt * 16 < tokens) nt *= 2;
  while (nt > 1 && tab + (size_t)nt * SP * 1024 + cols_bytes > kMaxLds) nt /= 2;
  const size_t slice = (size_t)nt * SP * 1024;
  if (tab + slice + cols_bytes > kMaxLds) return HL_EUNSUPPORTED;
  GemmArgs p;
  std::memset(&p, 0, sizeof(p));
  p.g = pl.ga;
  p.x = reinterpret_cast<const uint16_t*>(x_dev);
  p.y = y_dev;
  p.T = tokens;
  p.RS = gemm_row_sets(t);
  p.x_off = (uint32_t)slice;
  const uint32_t CB = pl.ga.CB;
  const uint32_t chunks = (tokens + 16 * nt - 1) / (16 * nt);
  // Column blocks per block: all of them when the row sets and chunks alone
  // give two blocks per CU; else split so that they do (one block fits a CU).
  const uint64_t base = (uint64_t)p.RS * chunks, target = 2ull * device_cus();
  p.cpb = base >= target ? CB : std::max<uint32_t>(1, (uint32_t)(CB * base / target));
  p.KS = (CB + p.cpb - 1) / p.cpb;
  p.partial = reinterpret_cast<float*>(workspace_dev);
  const uint64_t blocks = (uint64_t)p.KS * base;
  if (blocks >= (1ull << 31)) return HL_EUNSUPPORTED;
  const size_t lds = slice + cols_bytes;
  st = SP == 8 ? launch_gemm_sp<8>(nt, dim3((uint32_t)blocks), lds, (hipStream_t)stream, p)
               : launch_gemm_sp<4>(nt, dim3((uint32_t)blocks), lds, (hipStream_t)stream, p);
  if (st != HL_OK || p.KS == 1) return st;
  const uint64_t n = (uint64_t)tokens * t->rows;
  const uint32_t rblocks = (uint32_t)std::min<uint64_t>((n + 255) / 256, (uint64_t)device_cus() * 8);
  return launch(gemm_reduce_kernel, dim3(rblocks), dim3(256), 0, (hipStream_t)stream, p.partial, y_dev, p.KS, n);
}

extern "C" hl_status hl_gemv_bf16(const uint16_t* w_dev, uint64_t rows, uint64_t cols, const void* x_dev,
                                  hl_dtype x_dtype, uint32_t batch, float* y_dev, void* stream) {
  if (!w_dev || !x_dev || !y_dev || batch < 1 || batch > HL_MAX_BATCH || rows == 0 || cols == 0 ||
      cols % 8 || (x_dtype != HL_F32 && x_dtype != HL_BF16))
    return HL_EINVAL;
  if (!aligned(w_dev, 16) || !aligned(x_dev, 16) || !aligned(y_dev, 4)) return HL_EINVAL;
  if (rows >= (1ull << 31) || cols >= (1ull << 31)) return HL_EUNSUPPORTED;
  const uint32_t blocks = (uint32_t)std::min<uint64_t>((rows + 3) / 4, (uint64_t)device_cus() * 8);
  const bool xb = x_dtype == HL_BF16;
  HL_BATCH_SWITCH(launch_bf16_b, batch, xb, dim3(blocks), dim3(256), (hipStream_t)stream, w_dev, x_dev, y_dev,
                  (uint32_t)rows, (uint32_t)cols);
}
