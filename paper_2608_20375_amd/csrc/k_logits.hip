// k_logits.hip -- the logits pass: log-softmax statistics and top-K candidates
// of every drafter row q_{t,d} (the paper's Preliminaries, "DFlash one-pass
// marginals"; candidates = the highest-probability tokens of each position, as
// in the DDTree paragraph; conf_t of the SABA decoding state uses the top-1
// probability).
//
// One pass over the bf16 logits, HBM-bound.  Each workgroup (4 waves) streams
// one chunk of a row with 16-byte loads, 4 loads in flight per lane.  Each
// wave keeps an online softmax in log2 units: a wave-uniform offset mL (fp32,
// = max * log2 e) and per lane S = sum 2^y and T2 = sum 2^y * y with
// y = x * log2 e - mL, accumulated per tile in fp32 and across tiles in fp64.
// Top-K: every wave keeps a threshold (initially the K-th of the block's lane
// maxima over the first tiles, later the K-th value it has buffered, shared
// with the other waves); a tile whose maximum falls below it costs one
// ballot; a group of 8 values whose maximum reaches it is copied raw to a
// per-wave LDS ring, whose elements are offered to the wave's candidate
// buffer (ballot/mbcnt appends, a wave bitonic sort of (value desc, id asc)
// keys when full) only when the ring fills and at the end.  When there are
// too few rows to fill the chip, rows are split over several workgroups whose
// partial results a second small kernel merges.
#include "graft_internal.h"

namespace graft {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kUnroll = 4;                        // 16-byte loads per lane per tile
constexpr int kTileVec = kWave * kUnroll;         // 256 vectors = 2048 elements
constexpr float kL2E = 1.44269504088896340736f;
constexpr double kLn2 = 0.693147180559945309417232121458;
constexpr double kLog2e = 1.44269504088896340735992468100;
constexpr float kNegBig = -1e30f;                 // finite stand-in for -inf
constexpr int kTargetBlocks = 1024;                // one residency round at 4 waves/SIMD
constexpr int kMinSplitVec = 512;                 // >= 4096 elements per split
constexpr int kRing = 64;                         // deferred groups per wave

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

struct LaneStats {
  float mx;      // wave-uniform: largest logit the wave has seen
  float mL;      // wave-uniform fp32 offset: fl(mx * log2 e)
  double S;      // per lane: sum 2^(x*log2e - mL)
  double T2;     // per lane: sum 2^y * y
};

__device__ __forceinline__ void stats_init(LaneStats &s) {
  s.mx = kNegBig;
  s.mL = kNegBig * kL2E;
  s.S = 0.0;
  s.T2 = 0.0;
}

// Moves the wave's offset to its new maximum when some lane's value exceeds
// the old one, and rescales every lane's S and T2.  The factor
// 2^(mL_old - mL_new) is one v_exp_f32 of an fp32 difference (exact for offsets
// within a factor two of each other, and 0 for the initial finite stand-in).
__device__ __forceinline__ void stats_raise(LaneStats &s, float v) {
  if (__ballot(v > s.mx) == 0ull) return;
  float m = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) m = fmaxf(m, __uint_as_float(xor_lane(__float_as_uint(m), o)));
  m = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(m)));
  const float nL = m * kL2E;
  const float d = s.mL - nL;
  const double a = static_cast<double>(__builtin_amdgcn_exp2f(d));
  s.T2 = a * (s.T2 + static_cast<double>(d) * s.S);
  s.S = a * s.S;
  s.mL = nL;
  s.mx = m;
}

template <int CAP>
struct WaveBuf {
  uint64_t *buf;   // LDS [CAP]
  int count;       // wave-uniform
  float thr;       // wave-uniform: a candidate needs value >= thr
  uint4 *rq;       // LDS [kRing]: deferred groups of 8 raw bf16 values
  uint32_t *rid;   // LDS [kRing]: element id of each group's first value
  int rcount;      // wave-uniform
};

struct Compacted {
  int count;
  float thr;
};

// Sorts the first 64*E entries of a wave's buffer (count of them valid), keeps
// the best K keys and raises the threshold to the K-th value.  Out of line: it
// runs a few times per wave at most, and a single copy keeps the offer sites
// small.
template <int E>
__device__ __noinline__ Compacted compact_ool(uint64_t *buf, int count, float thr, int K) {
  const int lane = lane_id();
  uint64_t k[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = e * kWave + lane;
    k[e] = (i < count) ? buf[i] : 0ull;
  }
  wave_sort_desc<E>(k);
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = e * kWave + lane;
    if (i < K) buf[i] = k[e];
  }
  count = count < K ? count : K;
  if (count >= K) {
    const int src_e = (K - 1) / kWave, src_l = (K - 1) % kWave;
    uint64_t kth = 0;
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (e == src_e) kth = k[e];
    const uint32_t hi = __shfl(static_cast<uint32_t>(kth >> 32), src_l);
    const float t = unordered_f32(hi);
    thr = t > thr ? t : thr;
  }
  return {count, thr};
}

// Compaction sized to the number of buffered keys (K <= count rounded up).
template <int CAP>
__device__ __forceinline__ void wave_compact(WaveBuf<CAP> &w, int K) {
  const int need = w.count > K ? w.count : K;
  Compacted c;
  if (need <= kWave) c = compact_ool<1>(w.buf, w.count, w.thr, K);
  else if (need <= 2 * kWave || CAP == 2 * kWave) c = compact_ool<2>(w.buf, w.count, w.thr, K);
  else c = compact_ool<CAP / kWave>(w.buf, w.count, w.thr, K);
  // wave-uniform results: keep them in scalar registers
  w.count = __builtin_amdgcn_readfirstlane(c.count);
  w.thr = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(c.thr)));
}

// Offers one value per lane (valid lanes only) to the wave's buffer.
template <int CAP>
__device__ __forceinline__ void wave_offer(WaveBuf<CAP> &w, int K, float v, uint32_t id,
                                           bool valid) {
  bool pass = valid && v >= w.thr;
  uint64_t m = __ballot(pass);
  if (m == 0) return;
  int n = __popcll(m);
  if (w.count + n > CAP) {
    wave_compact<CAP>(w, K);
    pass = valid && v >= w.thr;
    m = __ballot(pass);
    if (m == 0) return;
    n = __popcll(m);
  }
  if (pass) w.buf[w.count + lanes_below(m)] = cand_key(v, id);
  w.count = __builtin_amdgcn_readfirstlane(w.count + n);
}

// Offers a 64-bit key per lane (used when merging already-sorted lists).
template <int CAP>
__device__ __forceinline__ void wave_offer_key(WaveBuf<CAP> &w, int K, uint64_t key) {
  const float v = cand_value(key);
  bool pass = key != 0ull && v >= w.thr;
  uint64_t m = __ballot(pass);
  if (m == 0) return;
  int n = __popcll(m);
  if (w.count + n > CAP) {
    wave_compact<CAP>(w, K);
    pass = key != 0ull && v >= w.thr;
    m = __ballot(pass);
    if (m == 0) return;
    n = __popcll(m);
  }
  if (pass) w.buf[w.count + lanes_below(m)] = key;
  w.count = __builtin_amdgcn_readfirstlane(w.count + n);
}

__device__ __forceinline__ void unpack8(const uint4 q, float (&v)[8]) {
  const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}

// Offers the deferred groups (one per lane) against the current threshold.
// A group was deferred when its largest value reached the threshold of the
// time; the threshold only rises, so comparing now drops nothing that belongs
// to the top K.  Out of line, with the buffer state passed by value.
template <int CAP>
__device__ __noinline__ Compacted flush_ool(uint64_t *buf, int count, float thr, const uint4 *rq,
                                            const uint32_t *rid, int rcount, int K) {
  const int lane = lane_id();
  WaveBuf<CAP> w{buf, count, thr, nullptr, nullptr, 0};
  const bool have = lane < rcount;
  uint4 r = make_uint4(0, 0, 0, 0);
  uint32_t id0 = 0;
  if (have) {
    r = rq[lane];
    id0 = rid[lane];
  }
  float v[8];
  unpack8(r, v);
  float gm = fmaxf(fmaxf(fmaxf(v[0], v[1]), v[2]), v[3]);
  gm = fmaxf(fmaxf(fmaxf(gm, v[4]), v[5]), fmaxf(v[6], v[7]));
  // The K-th largest group maximum is a lower bound of the wave's K-th value
  // (K distinct groups reach it): raise the threshold before offering.
  if (K <= kWave && rcount >= K) {
    uint32_t key[1] = {have ? ordered_f32(gm) : 0u};
    wave_sort_desc_u32<1>(key);
    const float tau = unordered_f32(__builtin_amdgcn_readlane(key[0], K - 1));
    if (tau > w.thr) w.thr = tau;
  }
  const bool live = have && gm >= w.thr;
  if (__ballot(live) != 0ull) {
#pragma unroll
    for (int e = 0; e < 8; ++e) wave_offer<CAP>(w, K, v[e], id0 + e, live);
  }
  return {w.count, w.thr};
}

// The last flush of a wave's ring, inlined so that every access stays an LDS
// access.  It first takes the largest threshold any wave of the block has
// published (each is a lower bound of the block's K-th value), then the K-th
// largest group maximum of the ring, and offers what survives both.
template <int CAP>
__device__ __forceinline__ void wave_flush_last(WaveBuf<CAP> &w, int K, const float *s_thr) {
  const int lane = lane_id();
  float o = w.thr;
#pragma unroll
  for (int i = 0; i < kWaves; ++i)
    o = fmaxf(o, __hip_atomic_load(&s_thr[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP));
  w.thr = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(o)));
  const bool have = lane < w.rcount;
  uint4 r = make_uint4(0, 0, 0, 0);
  uint32_t id0 = 0;
  if (have) {
    r = w.rq[lane];
    id0 = w.rid[lane];
  }
  float v[8];
  unpack8(r, v);
  float gm = fmaxf(fmaxf(fmaxf(v[0], v[1]), v[2]), v[3]);
  gm = fmaxf(fmaxf(fmaxf(gm, v[4]), v[5]), fmaxf(v[6], v[7]));
  if (K <= kWave && w.rcount >= K) {
    uint32_t key[1] = {have ? ordered_f32(gm) : 0u};
    wave_sort_desc_u32<1>(key);
    const float tau = unordered_f32(__builtin_amdgcn_readlane(key[0], K - 1));
    if (tau > w.thr) w.thr = tau;
  }
  const bool live = have && gm >= w.thr;
  if (__ballot(live) != 0ull) {
#pragma unroll
    for (int e = 0; e < 8; ++e) wave_offer<CAP>(w, K, v[e], id0 + e, live);
  }
  w.rcount = 0;
}

// Empties the wave's ring of deferred groups into its candidate buffer.
template <int CAP>
__device__ __forceinline__ void wave_flush(WaveBuf<CAP> &w, int K) {
  const Compacted c = flush_ool<CAP>(w.buf, w.count, w.thr, w.rq, w.rid, w.rcount, K);
  w.count = __builtin_amdgcn_readfirstlane(c.count);
  w.thr = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(c.thr)));
  w.rcount = 0;
}

// Loads one tile: lane handles vectors tile_vec + u*64 + lane, u < kUnroll.
template <bool MASKED>
__device__ __forceinline__ void load_tile(const uint4 *__restrict__ vec, int64_t tile_vec,
                                          int64_t n_vec, uint4 (&q)[kUnroll]) {
  const int lane = lane_id();
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const int64_t vi = tile_vec + u * kWave + lane;
    q[u] = make_uint4(0, 0, 0, 0);
    if (!MASKED || vi < n_vec) {
      const u32x4 x = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(vec) + vi);
      q[u] = make_uint4(x.x, x.y, x.z, x.w);
    }
  }
}

// One tile of loaded data: top-K candidates and softmax statistics.
template <int CAP, bool MASKED>
__device__ __forceinline__ void process_tile(const uint4 (&q)[kUnroll], int64_t tile_vec,
                                             int64_t n_vec, int64_t elem0, LaneStats &st,
                                             WaveBuf<CAP> &w, int K, float shared_thr) {
  const int lane = lane_id();
  float v[kUnroll][8];
  bool ok[kUnroll];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const int64_t vi = tile_vec + u * kWave + lane;
    ok[u] = !MASKED || vi < n_vec;
    unpack8(q[u], v[u]);
    if (MASKED && !ok[u]) {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[u][e] = kNegBig;
    }
  }
  // group maxima as chains of 3-input maxima (v_max3_f32)
  float sub[kUnroll];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const float a = fmaxf(fmaxf(v[u][0], v[u][1]), v[u][2]);
    const float b = fmaxf(fmaxf(a, v[u][3]), v[u][4]);
    const float c = fmaxf(fmaxf(b, v[u][5]), v[u][6]);
    sub[u] = fmaxf(c, v[u][7]);
  }
  const float tmax = fmaxf(fmaxf(fmaxf(sub[0], sub[1]), sub[2]), sub[3]);

  // top-K candidates; any wave's threshold bounds the block's K-th value.
  // A group of 8 whose largest value reaches the threshold is copied raw to
  // the wave's ring; the ring is offered element by element when it fills.
  if (shared_thr > w.thr) w.thr = shared_thr;
  if (__ballot(tmax >= w.thr) != 0ull) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const bool pass = ok[u] && sub[u] >= w.thr;
      const uint64_t m = __ballot(pass);
      if (m == 0ull) continue;
      const int n = __popcll(m);
      if (w.rcount + n > kRing) wave_flush<CAP>(w, K);
      if (pass) {
        const int slot = w.rcount + lanes_below(m);
        w.rq[slot] = q[u];
        w.rid[slot] = static_cast<uint32_t>(elem0 + (tile_vec + u * kWave + lane) * 8);
      }
      w.rcount = __builtin_amdgcn_readfirstlane(w.rcount + n);
    }
  }

  // softmax statistics
  stats_raise(st, tmax);
  const float mL = st.mL;
  // all arguments, then all exponentials, then the sums: no exp result is
  // consumed by the instruction right after it
  float s[kUnroll], t[kUnroll];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    float y[8], ex[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) y[e] = __builtin_fmaf(v[u][e], kL2E, -mL);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      ex[e] = __builtin_amdgcn_exp2f(y[e]);
      if (MASKED) ex[e] = ok[u] ? ex[e] : 0.f;
    }
    s[u] = ex[0];
    t[u] = ex[0] * y[0];
#pragma unroll
    for (int e = 1; e < 8; ++e) {
      s[u] += ex[e];
      t[u] = __builtin_fmaf(ex[e], y[e], t[u]);
    }
  }
  st.S += static_cast<double>((s[0] + s[1]) + (s[2] + s[3]));
  st.T2 += static_cast<double>((t[0] + t[1]) + (t[2] + t[3]));
}

// One vector per lane (valid lanes only): statistics and top-K candidates.
template <int CAP>
__device__ __forceinline__ void process_vec(const uint4 q, int64_t vi, bool valid, int64_t elem0,
                                            LaneStats &st, WaveBuf<CAP> &w, int K) {
  float v[8];
  unpack8(q, v);
  if (!valid) {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = kNegBig;
  }
  const float a = fmaxf(fmaxf(v[0], v[1]), v[2]);
  const float b = fmaxf(fmaxf(a, v[3]), v[4]);
  const float c = fmaxf(fmaxf(b, v[5]), v[6]);
  const float g = fmaxf(c, v[7]);
  const bool pass = valid && g >= w.thr;
  const uint64_t m = __ballot(pass);
  if (m != 0ull) {
    const int n = __popcll(m);
    if (w.rcount + n > kRing) wave_flush<CAP>(w, K);
    if (pass) {
      const int slot = w.rcount + lanes_below(m);
      w.rq[slot] = q;
      w.rid[slot] = static_cast<uint32_t>(elem0 + vi * 8);
    }
    w.rcount = __builtin_amdgcn_readfirstlane(w.rcount + n);
  }
  stats_raise(st, g);
  float s = 0.f, t = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float y = __builtin_fmaf(v[e], kL2E, -st.mL);
    const float ex = valid ? __builtin_amdgcn_exp2f(y) : 0.f;
    s += ex;
    t = __builtin_fmaf(ex, y, t);
  }
  st.S += static_cast<double>(s);
  st.T2 += static_cast<double>(t);
}

// One full tile with the block-shared threshold (other waves update their
// entries without a barrier; relaxed atomic reads keep the LDS addressing).
template <int CAP>
__device__ __forceinline__ void step_tile(const uint4 (&q)[kUnroll], int64_t t, int64_t n_vec,
                                          int64_t elem0, LaneStats &st, WaveBuf<CAP> &w, int K,
                                          float *s_thr, int wave) {
  float other = -INFINITY;
#pragma unroll
  for (int i = 0; i < kWaves; ++i)
    other = fmaxf(other, __hip_atomic_load(&s_thr[i], __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WORKGROUP));
  other = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(other)));
  const float before = w.thr;
  process_tile<CAP, false>(q, t * kTileVec, n_vec, elem0, st, w, K, other);
  if (lane_id() == 0 && w.thr > before)
    __hip_atomic_store(&s_thr[wave], w.thr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Scalar elements of a row that fall outside its 16-byte aligned body.
template <int CAP>
__device__ __forceinline__ void process_scalar(const uint16_t *__restrict__ row, int64_t idx,
                                               bool valid, LaneStats &st, WaveBuf<CAP> &w,
                                               int K) {
  float x = kNegBig;
  if (valid) x = __uint_as_float(static_cast<uint32_t>(row[idx]) << 16);
  wave_offer<CAP>(w, K, x, static_cast<uint32_t>(idx), valid);
  stats_raise(st, x);
  if (valid) {
    const float y = __builtin_fmaf(x, kL2E, -st.mL);
    const float ex = __builtin_amdgcn_exp2f(y);
    st.S += static_cast<double>(ex);
    st.T2 += static_cast<double>(ex * y);
  }
}

// Wave reduction of the per-lane sums (all lanes share the offset).
__device__ __forceinline__ void stats_wave_reduce(LaneStats &st) {
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    st.S += xor_lane_f64(st.S, o);
    st.T2 += xor_lane_f64(st.T2, o);
  }
}

// Merges (mL, S, T2) triples given with different offsets.
__device__ __forceinline__ void stats_merge(double &mL, double &S, double &T2, double mL2,
                                            double S2, double T22) {
  const double M = mL > mL2 ? mL : mL2;
  const double d1 = mL - M, d2 = mL2 - M;
  const double a1 = static_cast<double>(__builtin_amdgcn_exp2f(static_cast<float>(d1)));
  const double a2 = static_cast<double>(__builtin_amdgcn_exp2f(static_cast<float>(d2)));
  T2 = a1 * (T2 + d1 * S) + a2 * (T22 + d2 * S2);
  S = a1 * S + a2 * S2;
  mL = M;
}

struct RowOut {
  int32_t *ids;      // workspace [rows, K]
  float *logq;       // workspace [rows, K]
  float *stats;      // workspace [rows, 3]
  int32_t *o_ids;    // optional caller outputs
  float *o_logq, *o_lse, *o_maxprob, *o_ent;
};

// Final results of a row from merged statistics and the sorted top-K (wave 0).
template <int CAP>
__device__ __forceinline__ void write_row(const RowOut &o, int64_t row, int K, double mL,
                                          double S, double T2, const uint64_t *top) {
  const int lane = lane_id();
  // S >= 1 (the maximum contributes 2^0); the hardware log2 and exp2 in fp32
  // are accurate to about 2^-22 relative, far inside what the outputs need
  const double l2s = static_cast<double>(__builtin_amdgcn_logf(static_cast<float>(S)));
  const double lse2 = mL + l2s;
  const double lse = lse2 * kLn2;
  const double mx = static_cast<double>(cand_value(top[0]));
  for (int r = lane; r < K; r += kWave) {
    const uint64_t key = top[r];
    const int32_t id = key ? cand_id(key) : -1;
    const float lq = key ? static_cast<float>(static_cast<double>(cand_value(key)) - lse)
                         : -INFINITY;
    o.ids[row * K + r] = id;
    o.logq[row * K + r] = lq;
    if (o.o_ids) o.o_ids[row * K + r] = id;
    if (o.o_logq) o.o_logq[row * K + r] = lq;
  }
  if (lane == 0) {
    const float f_lse = static_cast<float>(lse);
    const float f_mp = __builtin_amdgcn_exp2f(static_cast<float>(mx * kLog2e - lse2));
    const float f_ent = static_cast<float>(kLn2 * (l2s - T2 / S));
    o.stats[row * 3 + 0] = f_lse;
    o.stats[row * 3 + 1] = f_mp;
    o.stats[row * 3 + 2] = f_ent;
    if (o.o_lse) o.o_lse[row] = f_lse;
    if (o.o_maxprob) o.o_maxprob[row] = f_mp;
    if (o.o_ent) o.o_ent[row] = f_ent;
  }
}

// Sorts the first n <= 64*E keys of buf (LDS) and writes the best K back to
// the front.
template <int E>
__device__ __forceinline__ void sort_front(uint64_t *buf, int n, int K) {
  const int lane = lane_id();
  uint64_t k[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = e * kWave + lane;
    k[e] = i < n ? buf[i] : 0ull;
  }
  wave_sort_desc<E>(k);
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = e * kWave + lane;
    if (i < K) buf[i] = k[e];
  }
}
template <int E>
__device__ __noinline__ void sort_front_ool(uint64_t *buf, int n, int K) {
  sort_front<E>(buf, n, K);
}

// Moves the keys of buf[from, n) that are larger than `above` to buf[to, ...)
// in order (to <= from: nothing is overwritten before it is read) and returns
// the new end.
__device__ __forceinline__ int keep_above(uint64_t *buf, int from, int n, int to,
                                          uint64_t above) {
  const int lane = lane_id();
  for (int j0 = from; j0 < n; j0 += kWave) {
    const int j = j0 + lane;
    const uint64_t key = j < n ? buf[j] : 0ull;
    const bool keep = j < n && key > above;
    const uint64_t b = __ballot(keep);
    if (keep) buf[to + lanes_below(b)] = key;
    to += __popcll(b);
  }
  return to;
}

// Top K of the block (wave 0).  Each wave's buffer holds keys at or above that
// wave's threshold, and the largest threshold is a lower bound of the block's
// K-th value: keys below it are dropped while the buffers are packed to the
// front of buf (a key never moves past an entry not yet read).  More than 256
// survivors are cut down by sorting the first 256 and keeping only keys above
// the K-th of those, which removes at least 256 - K keys per pass.  On return
// buf[0..K) holds the block's top K in descending key order, 0 past the last
// candidate.
template <int CAP>
__device__ __forceinline__ void block_merge(uint64_t *buf, const int *cnt, const float *thr,
                                            int K) {
  const int lane = lane_id();
  float th = thr[0];
#pragma unroll
  for (int i = 1; i < kWaves; ++i) th = fmaxf(th, thr[i]);
  int m = 0;
  for (int wv = 0; wv < kWaves; ++wv) {
    const int c = cnt[wv];
    for (int j0 = 0; j0 < c; j0 += kWave) {
      const int j = j0 + lane;
      const uint64_t key = j < c ? buf[wv * CAP + j] : 0ull;
      const bool keep = key != 0ull && cand_value(key) >= th;
      const uint64_t b = __ballot(keep);
      if (keep) buf[m + lanes_below(b)] = key;
      m += __popcll(b);
    }
  }
  while (m > 4 * kWave) {
    sort_front_ool<4>(buf, 4 * kWave, K);
    m = keep_above(buf, 4 * kWave, m, K, buf[K - 1]);
  }
  if (m <= kWave) sort_front<1>(buf, m, K);
  else if (m <= 2 * kWave) sort_front<2>(buf, m, K);
  else sort_front_ool<4>(buf, m, K);
  for (int i = m + lane; i < K; i += kWave) buf[i] = 0ull;
}

template <int CAP>
__global__ void __launch_bounds__(kThreads, 4)
logits_pass_kernel(const uint16_t *__restrict__ logits, int64_t V, int splits, int K,
                   double *__restrict__ part_stats, uint64_t *__restrict__ part_keys,
                   RowOut out) {
  __shared__ uint64_t s_buf[kWaves][CAP];
  __shared__ double s_stats[kWaves][3];
  __shared__ uint32_t s_init[kWaves * kMaxK];

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = lane_id();
  const int64_t row = blockIdx.x / splits;
  const int split = blockIdx.x % splits;

  const uint16_t *rowp = logits + row * V;
  // 16-byte aligned body of the row: elements [a0, a0 + 8 * nv_row)
  const int64_t abs0 = row * V;
  int64_t a0 = (8 - (abs0 & 7)) & 7;
  if (a0 > V) a0 = V;
  const int64_t nv_row = (V - a0) / 8;
  const int64_t per = (nv_row + splits - 1) / splits;
  const int64_t v_begin = per * split < nv_row ? per * split : nv_row;
  const int64_t v_end = v_begin + per < nv_row ? v_begin + per : nv_row;
  const int64_t n_vec = v_end - v_begin;
  const uint4 *vec = reinterpret_cast<const uint4 *>(rowp + a0) + v_begin;
  const int64_t elem0 = a0 + v_begin * 8;   // element id of vec[0]

  LaneStats st;
  stats_init(st);
  __shared__ uint4 s_rq[kWaves][kRing];
  __shared__ uint32_t s_rid[kWaves][kRing];
  WaveBuf<CAP> w{s_buf[wave], 0, -INFINITY, s_rq[wave], s_rid[wave], 0};

  // Tiles interleaved over the waves of the block; the next tile's loads are
  // issued before the current tile is processed.
  __shared__ float s_thr[kWaves];
  if (lane == 0) s_thr[wave] = -INFINITY;
  __syncthreads();
  const int64_t n_full = n_vec / kTileVec;
  int64_t t = wave;
  uint4 cur[kUnroll], nxt[kUnroll];
  const bool one = t < n_full, two = t + kWaves < n_full;
  if (one) {
    load_tile<false>(vec, t * kTileVec, n_vec, cur);
    load_tile<false>(vec, (two ? t + kWaves : t) * kTileVec, n_vec, nxt);
  }
  // The vectors past the full tiles (fewer than kTileVec) are spread over the
  // block, one per lane, and loaded with the first tiles; surplus lanes read
  // the last vector and are masked.
  const bool partial = n_full * kTileVec < n_vec;
  const int64_t pv = n_full * kTileVec + static_cast<int64_t>(wave) * kWave + lane;
  const bool pvalid = partial && pv < n_vec;
  uint4 extra = make_uint4(0, 0, 0, 0);
  if (partial) {
    const u32x4 x =
        __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(vec) + (pvalid ? pv : n_vec - 1));
    extra = make_uint4(x.x, x.y, x.z, x.w);
  }
  // Initial threshold, block wide: the K-th largest of the 256 lane maxima
  // over the waves' first two tiles.  K elements reach it, so it is a lower
  // bound of the row's K-th largest value.
  {
    float tm = kNegBig;
    if (one) {
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        float vv[8];
        unpack8(cur[u], vv);
#pragma unroll
        for (int e = 0; e < 8; ++e) tm = fmaxf(tm, vv[e]);
        if (two) {
          unpack8(nxt[u], vv);
#pragma unroll
          for (int e = 0; e < 8; ++e) tm = fmaxf(tm, vv[e]);
        }
      }
    }
    if (pvalid) {
      float vv[8];
      unpack8(extra, vv);
#pragma unroll
      for (int e = 0; e < 8; ++e) tm = fmaxf(tm, vv[e]);
    }
    uint32_t k1[1] = {ordered_f32(tm)};
    wave_sort_desc_u32<1>(k1);
    if (lane < K) s_init[wave * K + lane] = k1[0];
    __syncthreads();
    // the K-th of the union of the waves' K best (4 K <= CAP values)
    uint32_t kth;
    if (kWaves * K <= kWave) {
      uint32_t k2[1] = {lane < kWaves * K ? s_init[lane] : 0u};
      wave_sort_desc_u32<1>(k2);
      kth = __builtin_amdgcn_readlane(k2[0], K - 1);
    } else {
      constexpr int E2 = CAP / kWave;
      uint32_t k2[E2];
#pragma unroll
      for (int e = 0; e < E2; ++e) {
        const int i = e * kWave + lane;
        k2[e] = i < kWaves * K ? s_init[i] : 0u;
      }
      wave_sort_desc_u32<E2>(k2);
      const int src_e = (K - 1) / kWave;
      uint32_t v = 0;
#pragma unroll
      for (int e = 0; e < E2; ++e)
        if (e == src_e) v = k2[e];
      kth = __builtin_amdgcn_readlane(v, (K - 1) % kWave);
    }
    w.thr = unordered_f32(kth);
    if (w.thr < -1e29f) w.thr = -INFINITY;   // fewer than K real elements seen
  }
  if (partial) process_vec<CAP>(extra, pv, pvalid, elem0, st, w, K);
  if (one) {
    // ping-pong between two register buffers: the loads of tile t + kWaves are
    // in flight while tile t is processed
    // The prefetch of tile t + kWaves is issued on every step (past the last
    // tile it re-reads a valid one, a cache hit), so the wait before the
    // current tile covers only its own loads and never the prefetch.
    step_tile<CAP>(cur, t, n_vec, elem0, st, w, K, s_thr, wave);
    for (;;) {
      t += kWaves;
      if (t >= n_full) break;
      int64_t tl = t + kWaves < n_full ? t + kWaves : n_full - 1;
      load_tile<false>(vec, tl * kTileVec, n_vec, cur);
      step_tile<CAP>(nxt, t, n_vec, elem0, st, w, K, s_thr, wave);
      t += kWaves;
      if (t >= n_full) break;
      tl = t + kWaves < n_full ? t + kWaves : n_full - 1;
      load_tile<false>(vec, tl * kTileVec, n_vec, nxt);
      step_tile<CAP>(cur, t, n_vec, elem0, st, w, K, s_thr, wave);
    }
  }
  // Misaligned head [0, a0) and tail [a0 + 8 nv_row, V): split 0, wave 0.
  if (split == 0 && wave == 0) {
    const int64_t tail0 = a0 + 8 * nv_row;
    const int64_t n_head = a0, n_tail = V - tail0;
    if (n_head + n_tail > 0) {
      const bool valid = lane < n_head + n_tail;
      const int64_t idx = lane < n_head ? lane : tail0 + (lane - n_head);
      process_scalar<CAP>(rowp, valid ? idx : 0, valid, st, w, K);
    }
  }

  // Every wave's buffer stays unsorted: after one barrier wave 0 selects the
  // block's top K from all four at once.
  if (w.rcount > 0) wave_flush_last<CAP>(w, K, s_thr);
  stats_wave_reduce(st);
  __shared__ int s_cnt[kWaves];
  if (lane == 0) {
    s_stats[wave][0] = static_cast<double>(st.mL);
    s_stats[wave][1] = st.S;
    s_stats[wave][2] = st.T2;
    s_cnt[wave] = w.count;
    __hip_atomic_store(&s_thr[wave], w.thr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  __syncthreads();

  if (wave != 0) return;

  // Block merge in wave 0: statistics and the candidates of the four waves.
  double mL = s_stats[0][0], S = s_stats[0][1], T2 = s_stats[0][2];
  for (int i = 1; i < kWaves; ++i) stats_merge(mL, S, T2, s_stats[i][0], s_stats[i][1], s_stats[i][2]);
  block_merge<CAP>(&s_buf[0][0], s_cnt, s_thr, K);

  if (splits == 1) {
    write_row<CAP>(out, row, K, mL, S, T2, s_buf[0]);
    return;
  }

  // Split row: publish the partial; merge_kernel combines them after this
  // kernel has finished (the kernel boundary makes the writes visible).
  const int64_t slot = row * splits + split;
  for (int i = lane; i < K; i += kWave) part_keys[slot * K + i] = s_buf[0][i];
  if (lane == 0) {
    part_stats[slot * 3 + 0] = mL;
    part_stats[slot * 3 + 1] = S;
    part_stats[slot * 3 + 2] = T2;
  }
}

// One wave per split row: merges the partial statistics and top-K lists.
template <int CAP>
__global__ void __launch_bounds__(kWave)
merge_kernel(int splits, int K, const double *__restrict__ part_stats,
             const uint64_t *__restrict__ part_keys, RowOut out) {
  __shared__ uint64_t s_buf[CAP];
  const int64_t row = blockIdx.x;
  const int lane = lane_id();
  const double *ps = part_stats + row * splits * 3;
  double mL = ps[0], S = ps[1], T2 = ps[2];
  for (int i = 1; i < splits; ++i) stats_merge(mL, S, T2, ps[3 * i], ps[3 * i + 1], ps[3 * i + 2]);
  WaveBuf<CAP> m{s_buf, 0, -INFINITY, nullptr, nullptr, 0};
  const uint64_t *pk = part_keys + row * splits * K;
  const int total = splits * K;
  for (int base = 0; base < total; base += kWave) {
    const int i = base + lane;
    const uint64_t key = i < total ? pk[i] : 0ull;
    wave_offer_key<CAP>(m, K, key);
  }
  wave_compact<CAP>(m, K);
  for (int i = m.count + lane; i < K; i += kWave) s_buf[i] = 0ull;
  write_row<CAP>(out, row, K, mL, S, T2, s_buf);
}

}  // namespace

int logits_splits(const graft_dims &d, int rows) {
  const int64_t nv_row = d.vocab / 8;
  int64_t max_s = nv_row / kMinSplitVec;
  if (max_s < 1) max_s = 1;
  int64_t s = (kTargetBlocks + rows - 1) / rows;
  if (s > max_s) s = max_s;
  if (s < 1) s = 1;
  return static_cast<int>(s);
}

int logits_part_slots(const graft_dims &d) {
  int64_t best = 0;
  const int max_rows = d.max_batch * d.num_pos;
  for (int b = 1; b <= d.max_batch; ++b) {
    const int rows = b * d.num_pos;
    const int s = logits_splits(d, rows);
    if (s > 1 && static_cast<int64_t>(rows) * s > best) best = static_cast<int64_t>(rows) * s;
  }
  (void)max_rows;
  return static_cast<int>(best > 0 ? best : 1);
}

hipError_t launch_logits_pass(graft_ctx *ctx, const RoundScratch &ws, int batch,
                              const uint16_t *logits, const graft_tree_out *out,
                              hipStream_t stream) {
  const graft_dims &d = ctx->dims;
  const int rows = batch * d.num_pos;
  const int splits = logits_splits(d, rows);
  if (splits > 1 && static_cast<int64_t>(rows) * splits > ws.part_slots)
    return hipErrorInvalidValue;
  RowOut o;
  o.ids = ws.topk_ids;
  o.logq = ws.topk_logq;
  o.stats = ws.row_stats;
  o.o_ids = out ? out->topk_ids : nullptr;
  o.o_logq = out ? out->topk_logq : nullptr;
  o.o_lse = out ? out->row_lse : nullptr;
  o.o_maxprob = out ? out->row_maxprob : nullptr;
  o.o_ent = out ? out->row_entropy : nullptr;
  const dim3 grid(static_cast<unsigned>(rows * splits));
  const int64_t V = d.vocab;
  if (d.top_k <= 32) {
    hipLaunchKernelGGL(logits_pass_kernel<128>, grid, dim3(kThreads), 0, stream, logits, V,
                       splits, d.top_k, ws.part_stats, ws.part_keys, o);
    if (splits > 1)
      hipLaunchKernelGGL(merge_kernel<128>, dim3(rows), dim3(kWave), 0, stream, splits, d.top_k,
                         ws.part_stats, ws.part_keys, o);
  } else {
    hipLaunchKernelGGL(logits_pass_kernel<256>, grid, dim3(kThreads), 0, stream, logits, V,
                       splits, d.top_k, ws.part_stats, ws.part_keys, o);
    if (splits > 1)
      hipLaunchKernelGGL(merge_kernel<256>, dim3(rows), dim3(kWave), 0, stream, splits, d.top_k,
                         ws.part_stats, ws.part_keys, o);
  }
  return hipGetLastError();
}

}  // namespace graft
