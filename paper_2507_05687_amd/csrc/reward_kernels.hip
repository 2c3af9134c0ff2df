// Rule-based reward of the RL stage (AutoTriton Sec. 3.3, Eq. 3): a
// completion earns the reward when it is Triton code (is_Triton) and passed
// its tests (test_passed, an input from the execution harness); Sec. 4 names
// the rule (the @triton.jit decorator) and the hack of a decorated kernel
// that is never launched, which the optional launch check catches.
//
// The check is lexical, over the completion's bytes:
//   blank = space, tab or CR; identifier byte = [A-Za-z0-9_].
//   decorator: "@triton.jit" with only blanks before it on its line, not
//     followed by an identifier byte or "."; optional "(...)" arguments
//     (balanced, possibly over lines); then only blanks or a "#" comment
//     up to the newline.
//   decorated function: following blank, comment and decorator lines (a
//     decorator's parentheses balanced over lines) are skipped; the next line
//     must be: blanks, "def", blanks, a name not starting with a digit,
//     blanks, "(".
//   launch: the name, not preceded by an identifier byte, blanks, "[", a
//     bracket-balanced run to the matching "]", blanks, "(".
//
// One 256-thread workgroup per completion. A completion that fits (96 KiB)
// is first copied into LDS; its check costs a bounded amount of work per byte:
//   1. every thread tests 16 bytes in 4 KiB for a decorator; the functions
//      they decorate are followed up (by whole waves when there are few
//      decorators, else by the thread that found each) and their names go
//      into a hash table in LDS, each distinct name once;
//   2. a prefix-depth index of "[" / "]" over 32-byte chunks (depth at each
//      chunk's start, lowest depth within each chunk and each 1 KiB block)
//      lets a bracket find its match in at most a few hundred LDS reads;
//   3. every thread tests 16 bytes in 4 KiB for a "[" after an identifier
//      (and blanks) whose match is followed by blanks and "(" (a launch
//      site), and looks the identifier up in the table.
// is_Triton is an "exists" over decorators and launch sites, so the order in
// which threads find them does not change the result. A longer completion
// goes through the same passes reading the caller's text (never past
// text_bytes), with its name table in the idle LDS copy and index chunks of
// 32 bytes times ceil(length / 96 KiB), so a bracket match costs O(length /
// 3072) reads. More distinct decorated names than that table takes (6,144)
// are handled in rounds, each holding the names of one hash class; beyond 64
// rounds (some 390,000 names) the check falls back to simpler code: a name
// list and a text scan per name.
#include "kernels.h"

namespace grpo {
namespace {

// A completion: n bytes, in global memory (at t), or at base[i + sh] for
// byte i with base 16-byte aligned and cap bytes readable from it (the LDS
// copy, cap = its size; or the caller's text, cap = what is left of it), where
// long scans read 16 bytes at a time.
struct GlobalText {
  static constexpr bool kLds = false;
  const uint8_t* t;
  int64_t n;
  __device__ __forceinline__ uint8_t operator[](int64_t i) const { return t[i]; }
};
struct LdsText {
  static constexpr bool kLds = true;
  const uint8_t* base;
  int64_t sh;
  int64_t n;
  int64_t cap;
  __device__ __forceinline__ uint8_t operator[](int64_t i) const { return base[i + sh]; }
  // the 16 bytes at base + a (a multiple of 16); bytes at or past cap read as 0
  __device__ __forceinline__ u32x4 ld16(int64_t a) const {
    if (a + 16 <= cap) return *(const u32x4*)(base + a);
    u32x4 w = {0u, 0u, 0u, 0u};
    static_for<16>([&](auto k) {
      if (a + k.value < cap) w[k.value >> 2] |= (uint32_t)base[a + k.value] << (8 * (k.value & 3));
    });
    return w;
  }
};

__device__ __forceinline__ bool is_blank(uint8_t c) { return c == ' ' || c == '\t' || c == '\r'; }
__device__ __forceinline__ bool is_ident(uint8_t c) {
  return (c >= 'a' && c <= 'z') || (c >= 'A' && c <= 'Z') || (c >= '0' && c <= '9') || c == '_';
}

template <class T>
__device__ __forceinline__ int64_t skip_blanks(const T& X, int64_t i) {
  while (i < X.n && is_blank(X[i])) ++i;
  return i;
}

// 0x80 in each byte of x equal to v, 0 elsewhere
__device__ __forceinline__ uint32_t bytes_eq(uint32_t x, uint8_t v) {
  const uint32_t t = x ^ (0x01010101u * v);
  return ~(((t & 0x7f7f7f7fu) + 0x7f7f7f7fu) | t | 0x7f7f7f7fu);
}
__device__ __forceinline__ int count_eq(const u32x4& w, uint8_t v) {
  return __builtin_popcount(bytes_eq(w[0], v)) + __builtin_popcount(bytes_eq(w[1], v)) +
         __builtin_popcount(bytes_eq(w[2], v)) + __builtin_popcount(bytes_eq(w[3], v));
}

// index of the newline that ends the line holding i (or n). In LDS, whole
// 16-byte chunks without a newline are skipped at once.
template <class T>
__device__ __forceinline__ int64_t line_end(const T& X, int64_t i) {
  if constexpr (T::kLds) {
    for (; i < X.n && ((i + X.sh) & 15) != 0; ++i)
      if (X[i] == '\n') return i;
    for (; i + 16 <= X.n; i += 16) {
      const u32x4 w = X.ld16(i + X.sh);
      if (count_eq(w, '\n') != 0) break;
    }
  }
  while (i < X.n && X[i] != '\n') ++i;
  return i;
}

// X[i] opens a bracket pair (o, c): index just past its match, or -1. In
// LDS, a whole 16-byte chunk is skipped at once when its closing brackets
// cannot bring the depth to 0 (depth before it > closings in it).
template <class T>
__device__ __forceinline__ int64_t match_close(const T& X, int64_t i, uint8_t o, uint8_t c) {
  int64_t depth = 0;
  while (i < X.n) {
    if constexpr (T::kLds) {
      if (((i + X.sh) & 15) == 0 && i + 16 <= X.n && depth > 0) {
        const u32x4 w = X.ld16(i + X.sh);
        const int closes = count_eq(w, c);
        if (depth > closes) {
          depth += count_eq(w, o) - closes;
          i += 16;
          continue;
        }
      }
    }
    const uint8_t b = X[i];
    if (b == o) {
      ++depth;
    } else if (b == c) {
      if (--depth == 0) return i + 1;
    }
    ++i;
  }
  return -1;
}

// From i: an optional parenthesised run, then blanks or a comment to the
// newline. Start of the next line, or -1 if the line holds other text.
template <class T>
__device__ __forceinline__ int64_t finish_line(const T& X, int64_t i) {
  i = skip_blanks(X, i);
  if (i < X.n && X[i] == '(') {
    i = match_close(X, i, '(', ')');
    if (i < 0) return -1;
    i = skip_blanks(X, i);
  }
  if (i < X.n && X[i] != '\n' && X[i] != '#') return -1;
  return line_end(X, i) + 1;
}

constexpr char kDeco[] = "@triton.jit";
constexpr int kDecoLen = 11;

// a decorator starts at p (X[p] == '@' already known)
template <class T>
__device__ __forceinline__ bool decorator_at(const T& X, int64_t p) {
  if (p + kDecoLen > X.n) return false;
  for (int k = 1; k < kDecoLen; ++k)
    if (X[p + k] != (uint8_t)kDeco[k]) return false;
  const int64_t q = p + kDecoLen;
  if (q < X.n && (is_ident(X[q]) || X[q] == '.')) return false;
  for (int64_t j = p - 1; j >= 0 && X[j] != '\n'; --j)
    if (!is_blank(X[j])) return false;
  return true;
}

// name [ns, ns + nl) of the function decorated by the decorator at p.
// Also false when the follow-up reaches a later @triton.jit line whose own
// follow-up starts where this one continues: that decorator decorates the
// same function and reports it, so a stack of n decorators costs O(n) lines
// instead of O(n^2).
template <class T>
__device__ __forceinline__ bool decorated_name(const T& X, int64_t p, int64_t& ns, int64_t& nl) {
  int64_t i = finish_line(X, p + kDecoLen);
  while (i >= 0) {
    if (i >= X.n) return false;
    const int64_t j = skip_blanks(X, i);
    if (j >= X.n) return false;
    const uint8_t c = X[j];
    if (c == '\n' || c == '#') {  // blank or comment line
      i = line_end(X, j) + 1;
      continue;
    }
    if (c == '@') {  // another decorator
      int64_t k = j + 1;
      while (k < X.n && X[k] != '(' && X[k] != '\n') ++k;
      i = (k < X.n && X[k] == '(') ? finish_line(X, k) : line_end(X, k) + 1;
      if (i >= 0 && decorator_at(X, j) && finish_line(X, j + kDecoLen) == i) return false;
      continue;
    }
    if (!(j + 3 < X.n && X[j] == 'd' && X[j + 1] == 'e' && X[j + 2] == 'f' && is_blank(X[j + 3])))
      return false;
    int64_t k = skip_blanks(X, j + 3);
    if (k >= X.n || !is_ident(X[k]) || (X[k] >= '0' && X[k] <= '9')) return false;
    ns = k;
    while (k < X.n && is_ident(X[k])) ++k;
    nl = k - ns;
    k = skip_blanks(X, k);
    return k < X.n && X[k] == '(';
  }
  return false;
}

// a launch name[...]( of the name at [ns, ns + nl) starts at r
template <class T>
__device__ __forceinline__ bool launch_at(const T& X, int64_t r, int64_t ns, int64_t nl) {
  if (!(r + nl <= X.n && X[r] == X[ns] && (r == 0 || !is_ident(X[r - 1])))) return false;
  for (int64_t k = 1; k < nl; ++k)
    if (X[r + k] != X[ns + k]) return false;
  const int64_t s = skip_blanks(X, r + nl);
  if (!(s < X.n && X[s] == '[')) return false;
  int64_t e = match_close(X, s, '[', ']');
  if (e < 0) return false;
  e = skip_blanks(X, e);
  return e < X.n && X[e] == '(';
}

constexpr int kRrThreads = 256;
constexpr int kRrLds = 96 * 1024;  // completions up to this size (less 15 bytes) go to LDS
constexpr int kRrNames = 64;       // decorated functions listed per completion (global path)
constexpr int kRrList = 256;       // decorators followed up by whole waves (LDS path)
constexpr int kRrChunk = 32;                        // bytes per entry of the bracket index
constexpr int kRrChunks = kRrLds / kRrChunk;        // chunks of the longest LDS completion
constexpr int kRrBlock = 32;                        // chunks per block of the bracket index
constexpr int kRrBlocks = kRrChunks / kRrBlock;
// Name table slots: half again as many as the decorated functions a
// completion in LDS can hold (each takes at least "@triton.jit", a newline,
// "def ", one byte of name and "(", 18 bytes), so the table is at most two
// thirds full and probing always ends at an empty slot.
constexpr int kRrTable = 8192;
constexpr uint32_t kRrEmpty = 0xffffffffu;
static_assert(kRrLds / 18 * 3 / 2 < kRrTable && kRrLds < (1 << 17), "name table sizing");
constexpr int kRrTable64Max = kRrTable * 3 / 4;  // names a Table64 takes
static_assert(kRrTable * 8 <= kRrLds, "a Table64 lives in the idle LDS copy");

struct RrShared {
  int count;  // decorated functions found (may exceed kRrNames)
  int found;
  int overflow;  // a Table64 would take more than kRrTable64Max names
  int ntab;      // names a Table64 holds
  int nlist;  // entries of `list` found (may exceed kRrList)
  int64_t ns[kRrNames];
  int64_t nl[kRrNames];
  int64_t list[kRrList];
};

// Eq. 3's is_Triton for the completion X, the same in every thread of the
// workgroup; each thread follows up the decorators and launch candidates it
// finds by itself (global-memory completions, and lists that overflow).
template <class T>
__device__ __forceinline__ bool is_triton_block(const T& X, int require_launch, RrShared& sh) {
  const int tid = threadIdx.x;
  // phase 1: decorators and the functions they decorate
  for (int64_t base = 0; base < X.n; base += kRrThreads) {
    const int64_t p = base + tid;
    int64_t ns = 0, nl = 0;
    if (p < X.n && X[p] == '@' && decorator_at(X, p) && decorated_name(X, p, ns, nl)) {
      const int slot = atomicAdd(&sh.count, 1);
      if (slot < kRrNames) {
        sh.ns[slot] = ns;
        sh.nl[slot] = nl;
      }
    }
  }
  __syncthreads();
  const int count = sh.count;
  if (!require_launch || count == 0) return count > 0;
  if (count <= kRrNames) {
    // phase 2: a launch of any listed name
    for (int i = 0; i < count; ++i) {
      const int64_t ns = sh.ns[i], nl = sh.nl[i];
      for (int64_t base = 0; base < X.n; base += kRrThreads)
        if (__syncthreads_or(base + tid < X.n && launch_at(X, base + tid, ns, nl))) return true;
    }
    return false;
  }
  // too many to list: wave 0 takes the decorators in text order; a name equal
  // to one of the last kRecent names it found unlaunched is not searched again
  // (a completion that repeats one definition costs one search, not one per copy)
  if (tid < 64) {
    constexpr int kRecent = 4;
    int64_t rs[kRecent], rl[kRecent];
    static_for<kRecent>([&](auto q) { rs[q.value] = rl[q.value] = -1; });
    int next = 0;
    bool found = false;
    for (int64_t base = 0; base < X.n && !found; base += 64) {
      const int64_t p = base + tid;
      uint64_t m = __ballot(p < X.n && X[p] == '@' && decorator_at(X, p));
      while (m != 0 && !found) {
        const int64_t pp = base + (__ffsll((unsigned long long)m) - 1);
        m &= m - 1;
        int64_t ns = 0, nl = 0;
        if (!decorated_name(X, pp, ns, nl)) continue;
        bool seen = false;
        static_for<kRecent>([&](auto q) {
          if (!seen && rl[q.value] == nl) {
            bool eq = true;
            for (int64_t k = 0; k < nl && eq; ++k) eq = X[rs[q.value] + k] == X[ns + k];
            seen = eq;
          }
        });
        if (seen) continue;
        static_for<kRecent>([&](auto q) {
          if (q.value == next) {
            rs[q.value] = ns;
            rl[q.value] = nl;
          }
        });
        next = (next + 1) % kRecent;
        for (int64_t b2 = 0; b2 < X.n; b2 += 64) {
          if (__ballot(b2 + tid < X.n && launch_at(X, b2 + tid, ns, nl)) != 0) {
            found = true;
            break;
          }
        }
      }
    }
    if (tid == 0 && found) sh.found = 1;
  }
  __syncthreads();
  return sh.found != 0;
}

// ---- wave-cooperative scans over an LDS completion: every lane of the wave
// calls them with the same arguments and gets the same result; each lane
// takes one 16-byte chunk, 1 KiB per step.

// bit k set where byte k of the chunk w equals v
__device__ __forceinline__ uint32_t mask16(const u32x4& w, uint8_t v) {
  uint32_t r = 0;
  static_for<4>([&](auto d) {
    const uint32_t m = bytes_eq(w[d.value], v);
    r |= (((m >> 7) & 1) | ((m >> 14) & 2) | ((m >> 21) & 4) | ((m >> 28) & 8)) << (4 * d.value);
  });
  return r;
}
// bit k set where lo <= cs + k < hi
__device__ __forceinline__ uint32_t range16(int64_t cs, int64_t lo, int64_t hi) {
  const int64_t a = lo - cs > 0 ? lo - cs : 0, b = hi - cs < 16 ? hi - cs : 16;
  return b <= a ? 0u : ((1u << b) - 1u) & ~((1u << a) - 1u);
}

// first j >= i with X[j] equal to v1 or v2, else n
__device__ int64_t wave_find(const LdsText& X, int64_t i, uint8_t v1, uint8_t v2) {
  const int lane = threadIdx.x & 63;
  for (int64_t c0 = ((i + X.sh) & ~(int64_t)15) - X.sh; c0 < X.n; c0 += 1024) {
    const int64_t cs = c0 + 16 * lane;
    uint32_t hit = 0;
    if (cs < X.n && cs + 16 > i) {
      const u32x4 w = X.ld16(cs + X.sh);
      hit = (mask16(w, v1) | mask16(w, v2)) & range16(cs, i, X.n);
    }
    const uint64_t any = __ballot(hit != 0);
    if (any != 0) {
      const int l = __ffsll((unsigned long long)any) - 1;
      const int k = __shfl(hit != 0 ? __builtin_ctz(hit) : 0, l, 64);
      return c0 + 16 * l + k;
    }
  }
  return X.n;
}

// X[i] opens a bracket pair (o, c): index just past its match, or -1. Each
// lane takes the depth change and the lowest running depth of its chunk; a
// prefix sum over the wave gives the depth at each chunk's start, and the
// first chunk whose running depth reaches 0 holds the match.
__device__ int64_t wave_match_close(const LdsText& X, int64_t i, uint8_t o, uint8_t c) {
  const int lane = threadIdx.x & 63;
  int carry = 0;  // depth before this step's kibibyte
  for (int64_t c0 = ((i + X.sh) & ~(int64_t)15) - X.sh; c0 < X.n; c0 += 1024) {
    const int64_t cs = c0 + 16 * lane;
    int net = 0, low = 1 << 30;
    uint32_t mo = 0, mc = 0, valid = 0;
    if (cs < X.n && cs + 16 > i) {
      const u32x4 w = X.ld16(cs + X.sh);
      valid = range16(cs, i, X.n);
      mo = mask16(w, o) & valid;
      mc = mask16(w, c) & valid;
      static_for<16>([&](auto k) {
        net += (int)((mo >> k.value) & 1) - (int)((mc >> k.value) & 1);
        if ((valid >> k.value) & 1) low = net < low ? net : low;
      });
    }
    int incl = net;
    static_for<6>([&](auto s) {
      const int t = __shfl_up(incl, 1 << s.value, 64);
      if (lane >= (1 << s.value)) incl += t;
    });
    const int before = carry + incl - net;  // depth at the start of this lane's chunk
    const uint64_t any = __ballot(valid != 0 && before + low <= 0);
    if (any != 0) {
      const int l = __ffsll((unsigned long long)any) - 1;
      int at = 0;
      if (lane == l) {
        int d = before;
        for (int k = 0; k < 16; ++k) {
          d += (int)((mo >> k) & 1) - (int)((mc >> k) & 1);
          if (((valid >> k) & 1) && d == 0) {
            at = k;
            break;
          }
        }
      }
      return c0 + 16 * l + __shfl(at, l, 64) + 1;
    }
    carry += __shfl(incl, 63, 64);
  }
  return -1;
}

__device__ int64_t wave_line_end(const LdsText& X, int64_t i) { return wave_find(X, i, '\n', '\n'); }

__device__ int64_t wave_finish_line(const LdsText& X, int64_t i) {
  i = skip_blanks(X, i);
  if (i < X.n && X[i] == '(') {
    i = wave_match_close(X, i, '(', ')');
    if (i < 0) return -1;
    i = skip_blanks(X, i);
  }
  if (i < X.n && X[i] != '\n' && X[i] != '#') return -1;
  return wave_line_end(X, i) + 1;
}

// decorated_name with the long scans shared by the wave (used for at most
// kRrList decorators per completion, so it follows stacks to their end)
__device__ bool wave_decorated_name(const LdsText& X, int64_t p, int64_t& ns, int64_t& nl) {
  int64_t i = wave_finish_line(X, p + kDecoLen);
  while (i >= 0) {
    if (i >= X.n) return false;
    const int64_t j = skip_blanks(X, i);
    if (j >= X.n) return false;
    const uint8_t c = X[j];
    if (c == '\n' || c == '#') {
      i = wave_line_end(X, j) + 1;
      continue;
    }
    if (c == '@') {
      const int64_t k = wave_find(X, j + 1, '(', '\n');
      i = (k < X.n && X[k] == '(') ? wave_finish_line(X, k) : k + 1;
      continue;
    }
    if (!(j + 3 < X.n && X[j] == 'd' && X[j + 1] == 'e' && X[j + 2] == 'f' && is_blank(X[j + 3])))
      return false;
    int64_t k = skip_blanks(X, j + 3);
    if (k >= X.n || !is_ident(X[k]) || (X[k] >= '0' && X[k] <= '9')) return false;
    ns = k;
    while (k < X.n && is_ident(X[k])) ++k;
    nl = k - ns;
    k = skip_blanks(X, k);
    return k < X.n && X[k] == '(';
  }
  return false;
}

// ---- the LDS path's name table and bracket index

// A 16-byte aligned LDS chunk holding X[i] (i >= 0): its bytes, and the text
// index of its first byte.
__device__ __forceinline__ u32x4 lds_chunk(const LdsText& X, int64_t i, int64_t& c0) {
  const int64_t a = (i + X.sh) & ~(int64_t)15;
  c0 = a - X.sh;
  return X.ld16(a);
}
__device__ __forceinline__ uint8_t chunk_byte(const u32x4& w, int k) {
  return (uint8_t)(w[k >> 2] >> (8 * (k & 3)));
}

// skip_blanks reading 16 bytes at a time
__device__ int64_t lds_skip_blanks(const LdsText& X, int64_t i) {
  while (i < X.n) {
    int64_t c0;
    const u32x4 w = lds_chunk(X, i, c0);
    for (int k = (int)(i - c0); k < 16; ++k, ++i)
      if (i >= X.n || !is_blank(chunk_byte(w, k))) return i < X.n ? i : X.n;
  }
  return X.n;
}

// last index <= i holding a byte other than a blank, or -1, walking back 16
// bytes at a time
__device__ int64_t lds_back_skip_blanks(const LdsText& X, int64_t i) {
  while (i >= 0) {
    int64_t c0;
    const u32x4 w = lds_chunk(X, i, c0);
    for (int k = (int)(i - c0); k >= 0; --k, --i)
      if (c0 + k < 0 || !is_blank(chunk_byte(w, k))) return c0 + k < 0 ? -1 : i;
  }
  return -1;
}

// first byte of the identifier run that ends at r (X[r] is an identifier
// byte), walking back 16 bytes at a time
__device__ int64_t lds_ident_start(const LdsText& X, int64_t r) {
  int64_t i = r;
  while (i > 0) {
    int64_t c0;
    const u32x4 w = lds_chunk(X, i - 1, c0);
    for (int k = (int)(i - 1 - c0); k >= 0; --k, --i)
      if (c0 + k < 0 || !is_ident(chunk_byte(w, k))) return i;
  }
  return 0;
}

// FNV-1a hash of the identifier run [s, e)
__device__ uint32_t ident_hash(const LdsText& X, int64_t s, int64_t e) {
  uint32_t h = 2166136261u;
  int64_t i = s;
  while (i < e) {
    int64_t c0;
    const u32x4 w = lds_chunk(X, i, c0);
    for (int k = (int)(i - c0); k < 16 && i < e; ++k, ++i) h = (h ^ chunk_byte(w, k)) * 16777619u;
  }
  return h;
}

// the identifier runs starting at a and at b are equal
__device__ bool same_ident(const LdsText& X, int64_t a, int64_t b) {
  for (int64_t k = 0;; ++k) {
    const bool ia = a + k < X.n && is_ident(X[a + k]);
    const bool ib = b + k < X.n && is_ident(X[b + k]);
    if (ia != ib) return false;
    if (!ia) return true;
    if (X[a + k] != X[b + k]) return false;
  }
}

// Hash tables of the decorated names, one slot per distinct name. Table32
// (the LDS copy): a slot holds the position of the name's first byte (17
// bits) and 15 more bits of its hash; it has room for every name such a
// completion can hold. Table64 (longer completions): the position and the
// whole hash; it takes at most kRrTable64Max names and reports an overflow
// beyond that. kRrEmpty / ~0 mark free slots.
struct Table32 {
  uint32_t* s;
  __device__ void clear() const {
    for (int i = threadIdx.x; i < kRrTable; i += kRrThreads) s[i] = kRrEmpty;
  }
  __device__ bool insert(const LdsText& X, int64_t ns, uint32_t h, int*) const {
    const uint32_t v = (uint32_t)ns | ((h >> 13) << 17);
    for (uint32_t slot = h & (kRrTable - 1);; slot = (slot + 1) & (kRrTable - 1)) {
      const uint32_t old = atomicCAS(&s[slot], kRrEmpty, v);
      if (old == kRrEmpty) return true;
      if ((old >> 17) == (v >> 17) && same_ident(X, old & 0x1ffff, ns)) return true;
    }
  }
  __device__ bool find(const LdsText& X, int64_t st, uint32_t h) const {
    for (uint32_t slot = h & (kRrTable - 1);; slot = (slot + 1) & (kRrTable - 1)) {
      const uint32_t v = s[slot];
      if (v == kRrEmpty) return false;
      if ((v >> 17) == ((h >> 13) & 0x7fff) && same_ident(X, v & 0x1ffff, st)) return true;
    }
  }
};
struct Table64 {
  unsigned long long* s;
  __device__ void clear() const {
    for (int i = threadIdx.x; i < kRrTable; i += kRrThreads) s[i] = ~0ull;
  }
  // count: distinct names taken so far (shared); false once it would pass the limit
  __device__ bool insert(const LdsText& X, int64_t ns, uint32_t h, int* count) const {
    const unsigned long long v = ((unsigned long long)ns << 32) | h;
    for (uint32_t slot = h & (kRrTable - 1);; slot = (slot + 1) & (kRrTable - 1)) {
      const unsigned long long old = s[slot];
      if (old != ~0ull) {
        if ((uint32_t)old == h && same_ident(X, (int64_t)(old >> 32), ns)) return true;
        continue;
      }
      if (atomicAdd(count, 1) >= kRrTable64Max) return false;
      const unsigned long long got = atomicCAS(&s[slot], ~0ull, v);
      if (got == ~0ull) return true;
      atomicSub(count, 1);  // lost the slot to another name: look at it again
      slot = (slot - 1) & (kRrTable - 1);
    }
  }
  __device__ bool find(const LdsText& X, int64_t st, uint32_t h) const {
    for (uint32_t slot = h & (kRrTable - 1);; slot = (slot + 1) & (kRrTable - 1)) {
      const unsigned long long v = s[slot];
      if (v == ~0ull) return false;
      if ((uint32_t)v == h && same_ident(X, (int64_t)(v >> 32), st)) return true;
    }
  }
};

// The bracket index covers the text in chunks of C = 32 csub bytes aligned
// to base (chunk c holds text bytes C c - sh .. C c - sh + C - 1; bytes
// outside the text count as neither bracket). csub is 1 for the LDS copy and
// grows with a longer completion so that the index keeps kRrChunks entries.
struct BracketIndex {
  int32_t* cst;  // depth ("[" minus "]") before each chunk
  int32_t* cmn;  // lowest depth after any text byte of each chunk (2^30 if none)
  int32_t* bmn;  // lowest of cmn over each block of kRrBlock chunks
  int nch, nbl, csub;
};

__device__ __forceinline__ int bracket_step(uint8_t b) { return (b == '[') - (b == ']'); }

// Over the text bytes j of the 32-byte part at base + 32 u with from <= j < to,
// from depth d: the index just past the first byte after which the depth
// equals k, else -1 (d is then the depth after the last byte taken); lo
// tracks the lowest depth reached. The part is read into registers once.
__device__ __forceinline__ int64_t part_scan(const LdsText& X, int64_t u, int64_t from, int64_t to,
                                             int& d, int k, int& lo) {
  const u32x4 w0 = X.ld16(32 * u);
  const u32x4 w1 = X.ld16(32 * u + 16);
  const int64_t t0 = 32 * u - X.sh;
  if (from < 0) from = 0;
  if (to > X.n) to = X.n;
  int64_t hit = -1;
  static_for<32>([&](auto q) {
    const int64_t j = t0 + q.value;
    if (hit < 0 && j >= from && j < to) {
      d += bracket_step(chunk_byte(q.value < 16 ? w0 : w1, q.value & 15));
      lo = d < lo ? d : lo;
      if (d == k) hit = j + 1;
    }
  });
  return hit;
}

// Builds the index (all threads; ends with a barrier). Lane l of a row of 256
// takes chunk 256 row + l (consecutive chunks, free of bank conflicts in the
// LDS copy); depths are carried from row to row. wtot: 4 ints of LDS.
__device__ void build_bracket_index(const LdsText& X, BracketIndex& bi, int32_t* wtot) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t parts = (X.n + X.sh + 31) / 32;
  bi.csub = (int)((parts + kRrChunks - 1) / kRrChunks);
  bi.nch = (int)((parts + bi.csub - 1) / bi.csub);
  bi.nbl = (bi.nch + kRrBlock - 1) / kRrBlock;
  int carry = 0;  // depth before this row
  for (int row = 0; row * kRrThreads < bi.nch; ++row) {
    const int c = row * kRrThreads + tid;
    int net = 0, lo = 1 << 30;
    if (c < bi.nch)
      for (int p = 0; p < bi.csub; ++p)
        part_scan(X, (int64_t)c * bi.csub + p, 0, X.n, net, -(1 << 30), lo);
    int incl = net;  // inclusive scan within the wave
    static_for<6>([&](auto sft) {
      const int t = __shfl_up(incl, 1 << sft.value, 64);
      if (lane >= (1 << sft.value)) incl += t;
    });
    if (lane == 63) wtot[wave] = incl;
    __syncthreads();
    int before = carry + incl - net, total = 0;
    for (int v = 0; v < kRrThreads / 64; ++v) {
      before += v < wave ? wtot[v] : 0;
      total += wtot[v];
    }
    if (c < bi.nch) {
      bi.cst[c] = before;
      bi.cmn[c] = lo == (1 << 30) ? lo : before + lo;
    }
    carry += total;
    __syncthreads();
  }
  for (int b = tid; b < bi.nbl; b += kRrThreads) {
    int m = 1 << 30;
    const int e = (b + 1) * kRrBlock < bi.nch ? (b + 1) * kRrBlock : bi.nch;
    for (int c = b * kRrBlock; c < e; ++c) m = bi.cmn[c] < m ? bi.cmn[c] : m;
    bi.bmn[b] = m;
  }
  __syncthreads();
}

// Over the text bytes j of chunk c with from <= j < to: as part_scan
__device__ __forceinline__ int64_t chunk_find_depth(const LdsText& X, const BracketIndex& bi, int c,
                                                    int64_t from, int64_t to, int& d, int k) {
  int lo = 1 << 30;
  for (int p = 0; p < bi.csub; ++p) {
    const int64_t r = part_scan(X, (int64_t)c * bi.csub + p, from, to, d, k, lo);
    if (r >= 0) return r;
  }
  return -1;
}

// X[s] == '[': index just past its matching ']', or -1 (match_close's
// result). The match is the first byte after s where the depth returns to
// its value before s: found in s's chunk, else in the first later chunk of
// s's block, else of the first later block, whose lowest depth reaches it.
__device__ int64_t bracket_match(const LdsText& X, int64_t s, const BracketIndex& bi) {
  const int64_t C = 32 * (int64_t)bi.csub;
  const int c = (int)((s + X.sh) / C);
  int d = bi.cst[c];
  chunk_find_depth(X, bi, c, 0, s, d, -(1 << 30));  // the depth before s
  const int k = d++;  // the target depth; d is now the depth after s
  const int64_t r = chunk_find_depth(X, bi, c, s + 1, X.n, d, k);
  if (r >= 0) return r;
  const int be = (c / kRrBlock + 1) * kRrBlock < bi.nch ? (c / kRrBlock + 1) * kRrBlock : bi.nch;
  int cc = c + 1;
  while (cc < be && bi.cmn[cc] > k) ++cc;
  if (cc >= be) {
    int b = c / kRrBlock + 1;
    while (b < bi.nbl && bi.bmn[b] > k) ++b;
    if (b >= bi.nbl) return -1;
    cc = b * kRrBlock;
    while (bi.cmn[cc] > k) ++cc;  // some chunk of block b reaches k
  }
  d = bi.cst[cc];
  return chunk_find_depth(X, bi, cc, 0, X.n, d, k);  // found: cmn[cc] <= k
}

// is_Triton of a completion through the three bounded passes, the same in
// every thread: 1 or 0, or -1 when the names do not fit the table. If the
// decorated names overflow a Table64, the passes over names are repeated with
// the names split by hash: round j of k holds the names whose hash is j mod k
// and looks up only launch sites whose identifier hashes the same way (k is
// the decorated-function count over 4096, doubled while a round still
// overflows, at most kRrMaxRounds).
constexpr int kRrMaxRounds = 64;

template <class Table>
__device__ int is_triton_indexed(const LdsText& X, int require_launch, RrShared& sh,
                                 const Table& names, BracketIndex bi, int32_t* wtot) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  constexpr int kWaves = kRrThreads / 64;
  const int64_t nq = (X.n + X.sh + 15) / 16;  // 16-byte chunks from base
  bool indexed = false;
  for (int rounds = 1; rounds <= kRrMaxRounds;) {
    bool overflow = false;
    for (int j = 0; j < rounds && !overflow; ++j) {
      __syncthreads();  // the previous round is done with the table and the list
      if (tid == 0) {
        sh.count = 0;
        sh.nlist = 0;
        sh.overflow = 0;
        sh.ntab = 0;
      }
      names.clear();
      __syncthreads();
      auto add = [&](int64_t ns, int64_t nl) {  // a decorated function's name
        atomicAdd(&sh.count, 1);
        const uint32_t h = ident_hash(X, ns, ns + nl);
        if ((int)(h % (uint32_t)rounds) == j && !names.insert(X, ns, h, &sh.ntab)) sh.overflow = 1;
      };
      // 1. decorators; with at most kRrList of them the waves follow each up
      // (long scans shared by the wave), else the thread that found it does
      for (int64_t q = tid; q < nq; q += kRrThreads) {
        const int64_t t0 = 16 * q - X.sh;  // text index of the chunk's first byte
        uint32_t m = mask16(X.ld16(16 * q), '@') & range16(t0, 0, X.n);
        for (; m != 0; m &= m - 1) {
          const int64_t p = t0 + __builtin_ctz(m);
          if (decorator_at(X, p)) {
            const int slot = atomicAdd(&sh.nlist, 1);
            if (slot < kRrList) sh.list[slot] = p;
          }
        }
      }
      __syncthreads();
      const int ndeco = sh.nlist;
      if (ndeco <= kRrList) {
        for (int d = wave; d < ndeco; d += kWaves) {
          int64_t ns = 0, nl = 0;
          if (wave_decorated_name(X, sh.list[d], ns, nl) && lane == 0) add(ns, nl);
        }
      } else {
        for (int64_t q = tid; q < nq; q += kRrThreads) {
          const int64_t t0 = 16 * q - X.sh;
          uint32_t m = mask16(X.ld16(16 * q), '@') & range16(t0, 0, X.n);
          for (; m != 0; m &= m - 1) {
            const int64_t p = t0 + __builtin_ctz(m);
            int64_t ns = 0, nl = 0;
            if (decorator_at(X, p) && decorated_name(X, p, ns, nl)) add(ns, nl);
          }
        }
      }
      __syncthreads();
      if (!require_launch || sh.count == 0) return sh.count > 0;
      if (sh.overflow) {
        overflow = true;
        break;
      }
      // 2. the bracket index (once)
      if (!indexed) {
        build_bracket_index(X, bi, wtot);
        indexed = true;
      }
      // 3. launch sites and their names: each thread takes 16-byte chunks;
      // every "[" whose preceding non-blank byte ends an identifier is
      // matched through the index
      for (int64_t q0 = 0; q0 < nq; q0 += kRrThreads) {
        const int64_t q = q0 + tid;
        bool hit = false;
        if (q < nq) {
          const int64_t t0 = 16 * q - X.sh;  // text index of the chunk's first byte
          uint32_t m = mask16(X.ld16(16 * q), '[') & range16(t0, 0, X.n);
          while (m != 0 && !hit) {
            const int64_t s = t0 + __builtin_ctz(m);
            m &= m - 1;
            const int64_t r = lds_back_skip_blanks(X, s - 1);
            if (r < 0 || !is_ident(X[r])) continue;
            int64_t e = bracket_match(X, s, bi);
            if (e < 0) continue;
            e = lds_skip_blanks(X, e);
            if (e < X.n && X[e] == '(') {
              const int64_t st = lds_ident_start(X, r);
              const uint32_t h = ident_hash(X, st, r + 1);
              hit = (int)(h % (uint32_t)rounds) == j && names.find(X, st, h);
            }
          }
        }
        if (__syncthreads_or(hit)) return 1;
      }
    }
    if (!overflow) return 0;
    const int need = (sh.count + 4095) / 4096;
    rounds = need > 2 * rounds ? need : 2 * rounds;
  }
  return -1;
}

__global__ void __launch_bounds__(kRrThreads) k_rule_reward(RewardArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[kRrLds];
  __shared__ RrShared sh;
  __shared__ uint32_t names[kRrTable];
  __shared__ int32_t cst[kRrChunks], cmn[kRrChunks], bmn[kRrBlocks], wtot[kRrThreads / 64];
  const int64_t b = blockIdx.x;
  const int tid = threadIdx.x;
  // a pair outside [0, text_bytes] is an empty completion, like a decreasing one
  int64_t s0 = a.offsets[b], s1 = a.offsets[b + 1];
  if (s0 < 0 || s1 < 0 || s0 > a.text_bytes || s1 > a.text_bytes) s0 = s1 = 0;
  const int64_t n = s1 > s0 ? s1 - s0 : 0;
  if (tid == 0) {
    sh.count = 0;
    sh.found = 0;
    sh.nlist = 0;
    sh.overflow = 0;
    sh.ntab = 0;
  }
  bool found;
  // 16-byte aligned (text is), at most 15 bytes before s0
  const int64_t start = s0 & ~(int64_t)15;
  if (n + (s0 - start) <= kRrLds) {
    // copy [start, s1) to LDS: 16-byte loads up to the last whole 16 bytes
    // below s1, single bytes after that (nothing past s1 is read)
    const int64_t mid = n > 0 ? (s1 & ~(int64_t)15) : start;
    for (int64_t g = start + 16 * tid; g < mid; g += 16 * kRrThreads)
      *(u32x4*)(lds + (g - start)) = *(const u32x4*)(a.text + g);
    for (int64_t g = (mid > start ? mid : start) + tid; g < s1; g += kRrThreads)
      lds[g - start] = a.text[g];
    __syncthreads();
    found = is_triton_indexed(LdsText{lds, s0 - start, n, kRrLds}, a.require_launch, sh,
                              Table32{names}, BracketIndex{cst, cmn, bmn, 0, 0, 1}, wtot) > 0;
  } else {
    // longer than the copy: the same passes over the caller's text (read up
    // to text_bytes only), the name table in the idle copy; a completion
    // with more distinct names than that table takes falls back to the
    // simpler scan
    __syncthreads();
    int r = -1;
    if (n < (1ll << 31))
      r = is_triton_indexed(LdsText{a.text + start, s0 - start, n, a.text_bytes - start},
                            a.require_launch, sh, Table64{(unsigned long long*)lds},
                            BracketIndex{cst, cmn, bmn, 0, 0, 1}, wtot);
    if (r >= 0) {
      found = r > 0;
    } else {
      __syncthreads();
      if (tid == 0) {
        sh.count = 0;
        sh.found = 0;
        sh.nlist = 0;
      }
      __syncthreads();
      found = is_triton_block(GlobalText{a.text + s0, n}, a.require_launch, sh);
    }
  }
  if (tid == 0) {
    const bool passed = a.test_passed[b] != 0;
    a.is_triton[b] = found ? 1 : 0;
    a.reward[b] = a.weighted ? a.w_rule * (found ? 1.f : 0.f) + a.w_exec * (passed ? 1.f : 0.f)
                             : (found && passed ? 1.f : 0.f);
  }
}

}  // namespace

void launch_rule_reward(const RewardArgs& a, int64_t count, hipStream_t s) {
  hipLaunchKernelGGL(k_rule_reward, dim3((unsigned)count), dim3(kRrThreads), 0, s, a);
}

}  // namespace grpo
