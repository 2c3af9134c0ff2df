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
// One wave per completion. Lanes test 64 consecutive positions at a time for
// a decorator; each decorator found is followed up by the whole wave in text
// order (the function after it, then a launch search over the completion with
// one position per lane), so the result does not depend on timing.
#include "kernels.h"

namespace grpo {
namespace {

struct Text {
  const uint8_t* t;
  int64_t n;
};

__device__ __forceinline__ bool is_blank(uint8_t c) { return c == ' ' || c == '\t' || c == '\r'; }
__device__ __forceinline__ bool is_ident(uint8_t c) {
  return (c >= 'a' && c <= 'z') || (c >= 'A' && c <= 'Z') || (c >= '0' && c <= '9') || c == '_';
}

__device__ int64_t skip_blanks(const Text& T, int64_t i) {
  while (i < T.n && is_blank(T.t[i])) ++i;
  return i;
}

// index of the newline that ends the line holding i (or n)
__device__ int64_t line_end(const Text& T, int64_t i) {
  while (i < T.n && T.t[i] != '\n') ++i;
  return i;
}

// T.t[i] opens a bracket pair (o, c): index just past its match, or -1
__device__ int64_t match_close(const Text& T, int64_t i, uint8_t o, uint8_t c) {
  int64_t depth = 0;
  for (int64_t j = i; j < T.n; ++j) {
    if (T.t[j] == o) {
      ++depth;
    } else if (T.t[j] == c) {
      if (--depth == 0) return j + 1;
    }
  }
  return -1;
}

// From i: an optional parenthesised run, then blanks or a comment to the
// newline. Start of the next line, or -1 if the line holds other text.
__device__ int64_t finish_line(const Text& T, int64_t i) {
  i = skip_blanks(T, i);
  if (i < T.n && T.t[i] == '(') {
    i = match_close(T, i, '(', ')');
    if (i < 0) return -1;
    i = skip_blanks(T, i);
  }
  if (i < T.n && T.t[i] != '\n' && T.t[i] != '#') return -1;
  return line_end(T, i) + 1;
}

constexpr char kDeco[] = "@triton.jit";
constexpr int kDecoLen = 11;

// a decorator starts at p (T.t[p] == '@' already known)
__device__ bool decorator_at(const Text& T, int64_t p) {
  if (p + kDecoLen > T.n) return false;
  for (int k = 1; k < kDecoLen; ++k)
    if (T.t[p + k] != (uint8_t)kDeco[k]) return false;
  const int64_t q = p + kDecoLen;
  if (q < T.n && (is_ident(T.t[q]) || T.t[q] == '.')) return false;
  for (int64_t j = p - 1; j >= 0 && T.t[j] != '\n'; --j)
    if (!is_blank(T.t[j])) return false;
  return true;
}

// name [ns, ns + nl) of the function decorated by the decorator at p
__device__ bool decorated_name(const Text& T, int64_t p, int64_t& ns, int64_t& nl) {
  int64_t i = finish_line(T, p + kDecoLen);
  while (i >= 0) {
    if (i >= T.n) return false;
    const int64_t j = skip_blanks(T, i);
    if (j >= T.n) return false;
    const uint8_t c = T.t[j];
    if (c == '\n' || c == '#') {  // blank or comment line
      i = line_end(T, j) + 1;
      continue;
    }
    if (c == '@') {  // another decorator
      int64_t k = j + 1;
      while (k < T.n && T.t[k] != '(' && T.t[k] != '\n') ++k;
      i = (k < T.n && T.t[k] == '(') ? finish_line(T, k) : line_end(T, k) + 1;
      continue;
    }
    if (!(j + 3 < T.n && T.t[j] == 'd' && T.t[j + 1] == 'e' && T.t[j + 2] == 'f' &&
          is_blank(T.t[j + 3])))
      return false;
    int64_t k = skip_blanks(T, j + 3);
    if (k >= T.n || !is_ident(T.t[k]) || (T.t[k] >= '0' && T.t[k] <= '9')) return false;
    ns = k;
    while (k < T.n && is_ident(T.t[k])) ++k;
    nl = k - ns;
    k = skip_blanks(T, k);
    return k < T.n && T.t[k] == '(';
  }
  return false;
}

// some position holds name[...]( -- one position per lane, 64 at a time
__device__ bool launched(const Text& T, int64_t ns, int64_t nl, int lane) {
  for (int64_t base = 0; base < T.n; base += 64) {
    const int64_t r = base + lane;
    bool hit = false;
    if (r + nl <= T.n && T.t[r] == T.t[ns] && (r == 0 || !is_ident(T.t[r - 1]))) {
      bool eq = true;
      for (int64_t k = 1; k < nl && eq; ++k) eq = T.t[r + k] == T.t[ns + k];
      if (eq) {
        const int64_t s = skip_blanks(T, r + nl);
        if (s < T.n && T.t[s] == '[') {
          int64_t e = match_close(T, s, '[', ']');
          if (e >= 0) {
            e = skip_blanks(T, e);
            hit = e < T.n && T.t[e] == '(';
          }
        }
      }
    }
    if (__ballot(hit) != 0) return true;
  }
  return false;
}

__global__ void __launch_bounds__(64) k_rule_reward(RewardArgs a) {
  const int64_t b = blockIdx.x;
  const int lane = threadIdx.x;
  const int64_t s0 = a.offsets[b], s1 = a.offsets[b + 1];
  const Text T{a.text + s0, s1 > s0 ? s1 - s0 : 0};
  bool found = false;
  for (int64_t base = 0; base < T.n && !found; base += 64) {
    const int64_t p = base + lane;
    const bool cand = p < T.n && T.t[p] == '@' && decorator_at(T, p);
    uint64_t m = __ballot(cand);
    while (m != 0 && !found) {  // decorators of this stretch, in text order
      const int64_t pp = base + (__ffsll((unsigned long long)m) - 1);
      m &= m - 1;
      int64_t ns = 0, nl = 0;
      if (!decorated_name(T, pp, ns, nl)) continue;
      found = !a.require_launch || launched(T, ns, nl, lane);
    }
  }
  if (lane == 0) {
    const bool passed = a.test_passed[b] != 0;
    a.is_triton[b] = found ? 1 : 0;
    a.reward[b] = a.weighted ? a.w_rule * (found ? 1.f : 0.f) + a.w_exec * (passed ? 1.f : 0.f)
                             : (found && passed ? 1.f : 0.f);
  }
}

}  // namespace

void launch_rule_reward(const RewardArgs& a, int64_t count, hipStream_t s) {
  hipLaunchKernelGGL(k_rule_reward, dim3((unsigned)count), dim3(64), 0, s, a);
}

}  // namespace grpo
