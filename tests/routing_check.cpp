// Host-side check of the routing scorer (per-type argmin over the sorted
// instance table with the exact fp64 floor division and the migration rule,
// and the stateful variant that pins a future to the same-type instance
// holding its state).
// Random instance tables are laid out as the kernels lay them out (sorted by
// type, then index, with the run of each type), and route_future is compared
// with a plain integer argmin over every instance.  Cases cover random values, exact and near ties (equal loads,
// loads one apart), loads near 2^60 a few units of the last place apart,
// speeds near 2^31 and estimates near 2^40.
// Prints the number of mismatches.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <vector>
#include "common.hpp"

static uint64_t state = 0x2545F4914F6CDD1Dull;
static uint64_t next_rand() {  // splitmix64
  uint64_t z = (state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
static int64_t uni(int64_t lo, int64_t hi) {  // inclusive
  return lo + int64_t(next_rand() % uint64_t(hi - lo + 1));
}

struct Inst { int32_t type; int64_t load; int32_t speed; };

static void brute(const std::vector<Inst>& in, int32_t t, int64_t est, int32_t loc, int64_t mig,
                  bool stateful, int32_t& route, int64_t& cost) {
  if (stateful && loc >= 0 && in[loc].type == t) {
    route = loc;
    cost = in[loc].load + est * 1000 / in[loc].speed;
    return;
  }
  route = -1;
  cost = INT64_MAX;
  for (int i = 0; i < int(in.size()); ++i) {
    if (in[i].type != t) continue;
    const int64_t c = in[i].load + est * 1000 / in[i].speed + ((loc >= 0 && loc != i) ? mig : 0);
    if (c < cost) { cost = c; route = i; }
  }
}

static long long bad = 0, checked = 0;

static void run_case(const std::vector<Inst>& in, int n_types, int futures, int64_t est_max, int64_t mig) {
  const int M = int(in.size());
  std::vector<int> ord(M);
  for (int i = 0; i < M; ++i) ord[i] = i;
  std::stable_sort(ord.begin(), ord.end(), [&](int x, int y) { return in[x].type < in[y].type; });
  std::vector<int32_t> type(M), idx(M), speed(M), pos(M);
  std::vector<int64_t> load(M);
  std::vector<double> inv(M);
  std::vector<uint32_t> run(nalar::kTypeDirect, 0);
  for (int r = 0; r < M; ++r) {
    const Inst& x = in[ord[r]];
    type[r] = x.type; idx[r] = ord[r]; speed[r] = x.speed; load[r] = x.load;
    inv[r] = 1.0 / double(x.speed); pos[ord[r]] = r;
  }
  for (int r = 0; r < M; ++r) {
    const int t = type[r];
    if (t < nalar::kTypeDirect && (r == 0 || type[r - 1] != t)) {
      int e = r;
      while (e < M && type[e] == t) ++e;
      run[t] = uint32_t(r) | (uint32_t(e) << 16);
    }
  }
  for (int f = 0; f < futures; ++f) {
    const int32_t t = int32_t(uni(0, n_types - 1));
    int64_t est = uni(0, est_max);
    if (f % 7 == 0) est = est_max;
    const int32_t loc = (next_rand() & 1) ? int32_t(uni(0, M > 0 ? M - 1 : 0)) : -1;
    int32_t r0, r1;
    int64_t c0, c1;
    const bool stateful = (f % 3) == 1;
    brute(in, t, est, M > 0 ? loc : -1, mig, stateful, r0, c0);
    nalar::route_future(t, est, M > 0 ? loc : -1, M, mig, type.data(), idx.data(), load.data(),
                        speed.data(), inv.data(), pos.data(), run.data(), stateful, r1, c1);
    ++checked;
    if (r0 != r1 || c0 != c1) {
      if (bad < 10)
        std::printf("mismatch t=%d est=%lld loc=%d: route %d/%d cost %lld/%lld\n", t, (long long)est, loc,
                    r1, r0, (long long)c1, (long long)c0);
      ++bad;
    }
  }
}

int main() {
  const int64_t L60 = int64_t(1) << 60, E40 = int64_t(1) << 40;
  for (int rep = 0; rep < 3000; ++rep) {
    const int M = int(uni(1, 64));
    const int K = int(uni(1, 8));
    const int kind = rep % 7;
    std::vector<Inst> in(M);
    const int64_t base = uni(0, L60 - 4);
    const int32_t sp0 = int32_t(uni(1, 2000));
    const int64_t big = uni(L60 / 2, L60 - 1024);
    for (int i = 0; i < M; ++i) {
      Inst& x = in[i];
      x.type = int32_t(uni(0, K - 1));
      switch (kind) {
        case 0: x.load = uni(0, 2000000); x.speed = int32_t(uni(500, 2000)); break;      // the workloads
        case 1: x.load = 1000; x.speed = 1000; break;                                      // all equal
        case 2: x.load = 5000 + uni(0, 2); x.speed = sp0 + int32_t(uni(0, 1)); break;     // near ties
        case 3: x.load = base + uni(0, 3); x.speed = int32_t(uni(1, 3)); break;           // loads near 2^60
        case 4: x.load = uni(0, L60); x.speed = int32_t(uni(int64_t(1) << 30, (int64_t(1) << 31) - 1)); break;
        case 5: x.load = big + uni(0, 512); x.speed = int32_t(uni(500, 2000)); break;  // gaps of about one ulp
        default: x.load = uni(0, 1 << 20); x.speed = int32_t(uni(1, 1 << 16)); break;
      }
    }
    const int64_t est_max = kind == 5 ? 256 : kind == 3 || kind == 4 ? E40 : (rep % 2 ? E40 : 3000000);
    const int64_t mig = (rep % 3 == 0) ? 0 : (rep % 3 == 1 ? 200000 : uni(0, L60));
    run_case(in, K + 1, 64, est_max, mig);  // type K has no instance
  }
  std::printf("checked %lld mismatches %lld\n", checked, bad);
  return bad == 0 ? 0 : 1;
}
