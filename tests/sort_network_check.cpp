// Host check of the odd-even compare-exchange networks that the route
// kernel's top-k selection instantiates (csrc/sort_networks.hpp): every 0-1
// input of the 8- and 16-key sorts, every pair of sorted 0-1 runs for the
// 16 + 16 merge (by the 0-1 principle a comparator network that sorts these
// sorts every input), a sample of the 32-key sort's 0-1 inputs, random
// distinct keys, and the comparator counts.
#include <cstdio>
#include <cstdlib>

#include "sort_networks.hpp"

namespace {
int g_count = 0;
struct Cx {
  void operator()(int& a, int& b) const {
    ++g_count;
    if (a < b) {
      const int t = a;
      a = b;
      b = t;
    }
  }
};

int fails = 0;
void expect(bool ok, const char* what, unsigned case_id) {
  if (!ok && fails++ < 10) std::printf("FAIL %s case %u\n", what, case_id);
}
bool descending(const int* v, int lo, int hi) {
  for (int i = lo; i < hi; ++i)
    if (v[i] < v[i + 1]) return false;
  return true;
}
int ones(const int* v, int lo, int hi) {
  int n = 0;
  for (int i = lo; i <= hi; ++i) n += v[i];
  return n;
}
}  // namespace

int main() {
  for (unsigned m = 0; m < 256u; ++m) {
    int v[8];
    for (int i = 0; i < 8; ++i) v[i] = (m >> i) & 1;
    const int n1 = ones(v, 0, 7);
    mhl::oe_sort<0, 7>(v, Cx{});
    expect(descending(v, 0, 7) && ones(v, 0, 7) == n1, "sort 8", m);
  }
  for (unsigned m = 0; m < (1u << 16); ++m) {
    int v[16], w[16];
    for (int i = 0; i < 16; ++i) v[i] = w[i] = (m >> i) & 1;
    const int n1 = ones(v, 0, 15);
    mhl::oe_sort<0, 15>(v, Cx{});
    expect(descending(v, 0, 15) && ones(v, 0, 15) == n1, "sort 16", m);
    // the upper half sorted in place, the lower half untouched
    mhl::oe_sort<8, 15>(w, Cx{});
    bool lower_same = true;
    for (int i = 0; i < 8; ++i) lower_same &= w[i] == (int)((m >> i) & 1);
    expect(descending(w, 8, 15) && lower_same && ones(w, 8, 15) == ones(v, 0, 15) - ones(w, 0, 7),
           "sort 8..15", m);
  }
  for (int a = 0; a <= 16; ++a)
    for (int b = 0; b <= 16; ++b) {
      int v[32];
      for (int i = 0; i < 16; ++i) {
        v[i] = i < a;
        v[16 + i] = i < b;
      }
      mhl::oe_merge<0, 31, 1>(v, Cx{});
      expect(descending(v, 0, 31) && ones(v, 0, 31) == a + b, "merge 16+16", a * 17 + b);
    }
  std::srand(12345);
  for (unsigned r = 0; r < 2000; ++r) {
    int v[32];
    for (int i = 0; i < 32; ++i) v[i] = i;
    for (int i = 31; i > 0; --i) {
      const int j = std::rand() % (i + 1);
      const int t = v[i];
      v[i] = v[j];
      v[j] = t;
    }
    int s[16];
    for (int i = 0; i < 16; ++i) s[i] = v[i];
    mhl::oe_sort<0, 15>(s, Cx{});
    expect(descending(s, 0, 15), "random sort 16", r);
    mhl::oe_sort<0, 15>(v, Cx{});
    mhl::oe_sort<16, 31>(v, Cx{});
    mhl::oe_merge<0, 31, 1>(v, Cx{});
    bool perm_ok = true;
    for (int i = 0; i < 32; ++i) perm_ok &= v[i] == 31 - i;
    expect(perm_ok, "random merge", r);
  }
  // 32 keys (the paired-tile merge): 2^32 0-1 inputs are too many, so a
  // large random sample of them, every 0-1 input with at most two zeros or
  // two ones, and random permutations
  unsigned long long x = 88172645463325252ull;
  auto next = [&]() {
    x ^= x << 13;
    x ^= x >> 7;
    x ^= x << 17;
    return x;
  };
  for (unsigned r = 0; r < 300000; ++r) {
    int v[32];
    const unsigned long long m = next();
    for (int i = 0; i < 32; ++i) v[i] = (m >> i) & 1;
    const int n1 = ones(v, 0, 31);
    mhl::oe_sort<0, 31>(v, Cx{});
    expect(descending(v, 0, 31) && ones(v, 0, 31) == n1, "sort 32 random 0-1", r);
  }
  for (int a = 0; a < 32; ++a)
    for (int b = 0; b < 32; ++b)
      for (int bit = 0; bit < 2; ++bit) {
        int v[32];
        for (int i = 0; i < 32; ++i) v[i] = bit;
        v[a] = v[b] = 1 - bit;
        const int n1 = ones(v, 0, 31);
        mhl::oe_sort<0, 31>(v, Cx{});
        expect(descending(v, 0, 31) && ones(v, 0, 31) == n1, "sort 32 two-off", a * 64 + b * 2 + bit);
      }
  for (unsigned r = 0; r < 5000; ++r) {
    int v[32];
    for (int i = 0; i < 32; ++i) v[i] = i;
    for (int i = 31; i > 0; --i) {
      const int j = (int)(next() % (unsigned long long)(i + 1));
      const int t = v[i];
      v[i] = v[j];
      v[j] = t;
    }
    mhl::oe_sort<0, 31>(v, Cx{});
    bool ok = true;
    for (int i = 0; i < 32; ++i) ok &= v[i] == 31 - i;
    expect(ok, "sort 32 permutation", r);
  }
  int v[32] = {0};
  g_count = 0;
  mhl::oe_sort<0, 31>(v, Cx{});
  std::printf("comparators sort32 %d\n", g_count);
  expect(g_count == 191, "count sort 32", 0);
  g_count = 0;
  mhl::oe_sort<0, 7>(v, Cx{});
  std::printf("comparators sort8 %d\n", g_count);
  expect(g_count == 19, "count sort 8", 0);
  g_count = 0;
  mhl::oe_sort<0, 15>(v, Cx{});
  std::printf("comparators sort16 %d\n", g_count);
  expect(g_count == 63, "count sort 16", 0);
  g_count = 0;
  mhl::oe_merge<0, 31, 1>(v, Cx{});
  std::printf("comparators merge16+16 %d\n", g_count);
  expect(g_count == 65, "count merge", 0);
  std::printf("done %d failures\n", fails);
  return fails == 0 ? 0 : 1;
}
