// Stable LSD radix sort of (key, payload) pairs with one launch per 8-bit
// digit ("onesweep": a single upfront histogram of every digit, then each digit
// pass ranks its tile in LDS and finds its global offsets by decoupled
// look-back over earlier tiles, so no separate scan kernel is needed).
//
// Used twice per pass:
//  * the slack sort: key = slack - min slack (range-reduced, so only the digits
//    the key range needs are sorted), payload = position of the ready future;
//    its first pass reads the futures staged by position and skips the
//    positions that are not ready, so it also compacts them, and the stable
//    passes keep (wf, id) order among equal slacks;
//  * grouping futures by workflow when the caller's ids are not grouped:
//    key = wf, payload = id.
//
// Tile layout: 256 threads (4 waves), 16 items per thread, wave w owning a
// contiguous run of 1024 items with item j of lane l at offset j*64 + l, so
// loads are coalesced and the in-wave ranking visits items in input order.
#include "internal.hpp"

namespace nalar {

namespace {

constexpr int kWavesPerTile = kSortThreads / kWave;

template <typename K>
__device__ inline K first_key(const RadixDesc& d, int src, int64_t i, int64_t slack_min) {
  if (src == kSrcStaged) return K(uint64_t(d.stg_slack[i] - slack_min));
  return K(uint32_t(d.wf[i]));
}

__device__ inline bool first_valid(const RadixDesc& d, int src, int64_t i) {
  return i < d.first_span && (src != kSrcStaged || d.stg_ready[i] != 0);
}

// Slack range and ready count of the staged futures, from the sweep's slots.
struct StagedRange {
  int64_t smin, smax, count;
};

__device__ inline StagedRange reduce_parts(const Ctrl* ctrl) {
  StagedRange r{INT64_MAX, INT64_MIN, 0};
  for (int i = 0; i < kParts; ++i) {
    const int64_t a = ctrl->part_min[i], b = ctrl->part_max[i];
    r.smin = a < r.smin ? a : r.smin;
    r.smax = b > r.smax ? b : r.smax;
    r.count += ctrl->part_cnt[i];
  }
  return r;
}

// Digit histograms of all passes the key range needs.  For the slack sort this
// kernel also settles the ready count, the slack range and the pass count
// (at least one pass when anything is ready: the first pass compacts).
template <typename K>
__global__ __launch_bounds__(kSortThreads) void k_radix_hist(RadixDesc d, Ctrl* ctrl, int src) {
  if (ctrl->status) return;
  int npass;
  int64_t smin = 0;
  if (d.npass_host < 0) {
    const StagedRange r = reduce_parts(ctrl);
    smin = r.smin;
    int nbits = 0;
    if (r.count > 0) {
      const uint64_t range = uint64_t(r.smax - r.smin);
      nbits = range ? 64 - __builtin_clzll(range) : 0;
    }
    npass = r.count > 0 ? (nbits + kRadixBits - 1) / kRadixBits : 0;
    if (r.count > 0 && npass == 0) npass = 1;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      ctrl->slack_min = r.smin;
      ctrl->slack_max = r.smax;
      ctrl->n_ready = r.count;
      ctrl->sort_npass = uint32_t(npass);
    }
  } else {
    npass = d.npass_host;
  }
  if (npass == 0) return;
  __shared__ uint32_t h[kMaxSortPasses][kRadixBuckets];
  for (int i = threadIdx.x; i < kMaxSortPasses * kRadixBuckets; i += kSortThreads)
    (&h[0][0])[i] = 0;
  __syncthreads();
  const int64_t span = d.first_span;
  const int64_t stride = int64_t(gridDim.x) * kSortThreads;
  for (int64_t base = int64_t(blockIdx.x) * kSortThreads; base < span; base += stride) {
    const int64_t i = base + threadIdx.x;
    const bool valid = first_valid(d, src, i);
    const K key = valid ? first_key<K>(d, src, i, smin) : K(0);
    for (int ps = 0; ps < npass; ++ps) {
      const uint32_t dg = uint32_t(key >> (ps * kRadixBits)) & (kRadixBuckets - 1);
      // most high digits are shared by the whole wave: one add instead of 64
      const uint64_t act = ballot(valid);
      const int first = readlane_i32(int(dg), act ? __builtin_ctzll(act) : 0);
      const uint64_t same = ballot(valid && int(dg) == first);
      if (same == act) {
        if (act && lane_id() == __builtin_ctzll(act)) atomicAdd(&h[ps][dg], uint32_t(__popcll(act)));
      } else if (valid) {
        atomicAdd(&h[ps][dg], 1u);
      }
    }
  }
  __syncthreads();
  for (int ps = 0; ps < npass; ++ps)
    for (int b = threadIdx.x; b < kRadixBuckets; b += kSortThreads)
      if (h[ps][b]) atomicAdd(&d.ghist[ps * kRadixBuckets + b], h[ps][b]);
}

// Exclusive scan of one value per thread over the 256-thread block.
__device__ inline uint32_t block_excl_scan(uint32_t x, uint32_t* s_tmp) {
  const int w = threadIdx.x / kWave;
  const uint32_t inc = wave_incl_scan_u32(x);
  if (lane_id() == kWave - 1) s_tmp[w] = inc;
  __syncthreads();
  uint32_t off = 0;
  for (int i = 0; i < w; ++i) off += s_tmp[i];
  __syncthreads();
  return off + inc - x;
}

template <typename K>
__global__ __launch_bounds__(kSortThreads) void k_radix_pass(RadixDesc d, Ctrl* ctrl, int src,
                                                             int pass, uint32_t epoch) {
  if (ctrl->status) return;
  const int npass = d.npass_host >= 0 ? d.npass_host : int(ctrl->sort_npass);
  if (pass >= npass) return;
  const bool first = pass == 0 && src != kSrcBuffers;
  const int64_t R = d.count_dev ? *d.count_dev : d.count_host;   // dense count
  const int64_t span = first ? d.first_span : R;                  // items scanned
  const int64_t ntiles = (span + kSortTile - 1) / kSortTile;

  __shared__ uint32_t s_tile;
  __shared__ uint32_t s_whist[kWavesPerTile][kRadixBuckets];
  __shared__ uint32_t s_tprefix[kRadixBuckets];
  __shared__ uint64_t s_gstart[kRadixBuckets];
  __shared__ uint32_t s_tmp[kWavesPerTile];
  __shared__ uint32_t s_intile;
  __shared__ K s_key[kSortTile];
  __shared__ uint32_t s_pay[kSortTile];

  const int tid = threadIdx.x;
  if (tid == 0) s_tile = atomicAdd(&ctrl->tile_ticket[d.ticket_base + pass], 1u);
  for (int i = tid; i < kWavesPerTile * kRadixBuckets; i += kSortThreads) (&s_whist[0][0])[i] = 0;
  __syncthreads();
  const int64_t tile = s_tile;
  if (tile >= ntiles) return;

  const int wv = tid / kWave;
  const int ln = lane_id();
  const int shift = pass * kRadixBits;
  const int64_t seg = tile * kSortTile + int64_t(wv) * (kWave * kSortItems);
  const int64_t smin = (src == kSrcStaged) ? ctrl->slack_min : 0;
  const K* kin = static_cast<const K*>(d.key_buf[(pass + 1) & 1]);
  const uint32_t* pin = d.pay_buf[(pass + 1) & 1];
  K* kout = static_cast<K*>(d.key_buf[pass & 1]);
  uint32_t* pout = d.pay_buf[pass & 1];

  K key[kSortItems];
  uint32_t pay[kSortItems];
  uint32_t rank[kSortItems];
  uint32_t validm = 0;
#pragma unroll
  for (int j = 0; j < kSortItems; ++j) {
    const int64_t i = seg + j * kWave + ln;
    key[j] = K(0);
    pay[j] = 0;
    if (first) {
      if (first_valid(d, src, i)) {
        key[j] = first_key<K>(d, src, i, smin);
        pay[j] = uint32_t(i);
        validm |= 1u << j;
      }
    } else if (i < span) {
      key[j] = kin[i];
      pay[j] = pin[i];
      validm |= 1u << j;
    }
  }

  // In-wave stable ranking: lanes with equal digits found by 8 ballots; the
  // per-wave running count of each digit lives in LDS.
  uint32_t* wh = s_whist[wv];
#pragma unroll
  for (int j = 0; j < kSortItems; ++j) {
    const bool valid = (validm >> j) & 1u;
    const uint32_t dg = uint32_t(key[j] >> shift) & (kRadixBuckets - 1);
    uint64_t peers = ballot(valid);
#pragma unroll
    for (int b = 0; b < kRadixBits; ++b) {
      const bool bit = (dg >> b) & 1u;
      const uint64_t m = ballot(bit);
      peers &= bit ? m : ~m;
    }
    const uint64_t below = peers & lanemask_lt();
    uint32_t cnt = 0;
    if (valid) cnt = wh[dg];
    rank[j] = cnt + uint32_t(__popcll(below));
    if (valid && below == 0) wh[dg] = cnt + uint32_t(__popcll(peers));
  }
  __syncthreads();

  // Digit totals of the tile; per-wave counts become exclusive offsets.
  const int dg = tid;  // 256 threads, 256 digits
  uint32_t tot = 0;
#pragma unroll
  for (int w = 0; w < kWavesPerTile; ++w) {
    const uint32_t c = s_whist[w][dg];
    s_whist[w][dg] = tot;
    tot += c;
  }
  uint64_t* lb = d.lookback + (int64_t(pass) * d.tiles_cap) * kRadixBuckets + dg;
  st_relaxed_agent(lb + tile * kRadixBuckets, lb_pack(epoch, tile == 0 ? kLbInc : kLbAgg, tot));
  const uint32_t gh = d.ghist[pass * kRadixBuckets + dg];
  const uint32_t gexcl = block_excl_scan(gh, s_tmp);
  const uint32_t texcl = block_excl_scan(tot, s_tmp);
  uint64_t excl = 0;
  if (tile > 0) {
    excl = lookback_exclusive(lb, tile, kRadixBuckets, epoch);
    st_relaxed_agent(lb + tile * kRadixBuckets, lb_pack(epoch, kLbInc, excl + tot));
  }
  s_tprefix[dg] = texcl;
  s_gstart[dg] = uint64_t(gexcl) + excl;
  if (dg == kRadixBuckets - 1) s_intile = texcl + tot;
  __syncthreads();

  // Stage the tile in digit order in LDS, then write runs of equal digits to
  // consecutive global addresses.
#pragma unroll
  for (int j = 0; j < kSortItems; ++j) {
    if ((validm >> j) & 1u) {
      const uint32_t dgt = uint32_t(key[j] >> shift) & (kRadixBuckets - 1);
      const uint32_t pos = s_tprefix[dgt] + s_whist[wv][dgt] + rank[j];
      s_key[pos] = key[j];
      s_pay[pos] = pay[j];
    }
  }
  __syncthreads();
  const int in_tile = int(s_intile);
  for (int i = tid; i < in_tile; i += kSortThreads) {
    const K k = s_key[i];
    const uint32_t dgt = uint32_t(k >> shift) & (kRadixBuckets - 1);
    const uint64_t g = s_gstart[dgt] + uint64_t(i - int(s_tprefix[dgt]));
    if (g < uint64_t(R)) {
      kout[g] = k;
      pout[g] = s_pay[i];
    }
  }
}

int hist_grid(int64_t n) {
  int64_t b = (n + kSortTile - 1) / kSortTile;
  if (b < 1) b = 1;
  if (b > 2048) b = 2048;
  return int(b);
}

}  // namespace

hipError_t launch_radix_hist(hipStream_t s, const RadixDesc& d, Ctrl* ctrl, int src,
                             int64_t max_count, bool key64) {
  if (key64)
    hipLaunchKernelGGL(k_radix_hist<uint64_t>, dim3(hist_grid(max_count)), dim3(kSortThreads), 0,
                       s, d, ctrl, src);
  else
    hipLaunchKernelGGL(k_radix_hist<uint32_t>, dim3(hist_grid(max_count)), dim3(kSortThreads), 0,
                       s, d, ctrl, src);
  return hipGetLastError();
}

hipError_t launch_radix_pass(hipStream_t s, const RadixDesc& d, Ctrl* ctrl, int src, int pass,
                             uint32_t epoch, int64_t max_count, bool key64) {
  int64_t tiles = (max_count + kSortTile - 1) / kSortTile;
  if (tiles < 1) tiles = 1;
  if (key64)
    hipLaunchKernelGGL(k_radix_pass<uint64_t>, dim3(unsigned(tiles)), dim3(kSortThreads), 0, s, d,
                       ctrl, src, pass, epoch);
  else
    hipLaunchKernelGGL(k_radix_pass<uint32_t>, dim3(unsigned(tiles)), dim3(kSortThreads), 0, s, d,
                       ctrl, src, pass, epoch);
  return hipGetLastError();
}

}  // namespace nalar
