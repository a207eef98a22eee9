// Single-pass window statistics: row softmax statistics and per-token mean / dispersion
// (section 3.1, Eq. (1), Eq. (3)) reading every cached key once, for bf16 caches with w = 32.
//
// The row normaliser of a window query needs every key of its (problem, kv head) "unit" before any
// token's attention can be formed.  Each workgroup therefore keeps the keys it has scored on chip
// until its unit's normalisers are known, and forms the attention from them a second time:
//
//   item = 256 keys of one unit (8 waves x one 32-key MFMA tile).  Items are dealt round-robin to
//   the persistent workgroups, so a unit's items run side by side on many workgroups.  Each
//   workgroup pipelines its items through four register slots:
//
//     iteration i:  phase 1 of item i     logits D[key][row] = K Q^T (v_mfma_f32_32x32x16_bf16, keys
//                                         as M so that a lane holds one window row), per-wave row
//                                         maximum m and sum z of 2^(t - m), merged over the waves;
//                                         the item's partial (m, z) per row is stored for its unit
//                                         (write-through store, nothing waited for);
//                   phase 2 of item i-2   the unit's normalisers b = M + log2 Z are known by now:
//                                         logits again with keys as N (a lane holds one key),
//                                         a = 2^(t - b) summed over the group's heads, then the mean
//                                         and the two-pass sample variance over the window rows;
//                   keys of item i+2 are requested into the slot item i-2 has just released.
//
//   The merge is spread over the unit's items: the last M = min(n, R, grid) of its n items own the
//   window rows r = c - (n - M) (mod M) each.  One iteration after publishing item c, its
//   workgroup polls every item's partial of the rows it owns (initialised to a NaN sentinel),
//   combines them and stores those rows' normalisers and row_max / row_sum outputs.  The
//   normalisers of item i - 2's unit are requested at the end of iteration i - 1 and waited for
//   in iteration i.  Exchanged values use device-scope accesses, which bypass the per-XCD caches;
//   every wait is bounded.
//
// Deadlock freedom (n <= grid, checked at launch, so that a workgroup holds at most one item of
// a unit and the items of a unit lie in consecutive iterations of the workgroups): iteration j of
// every workgroup publishes item j, then merges for item j - 1, then waits for item j - 2's unit.
// Take the smallest iteration j at which some workgroup waits.  The other items of item j - 1's
// unit lie at iterations <= j of their workgroups, all already published; the owners of item
// j - 2's rows lie at iterations <= j - 1 and have merged by iteration j, before their own wait.
// So every wait at iteration j ends.  The grid is launched cooperatively so that every workgroup
// is resident.
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace kv {

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
constexpr int kItemKeys = kWaves * 32;  // keys per item
static_assert(kItemKeys == kFusedChunk, "an item is one chunk");
constexpr int kSlots = 4;   // register slots of key tiles per wave
constexpr int kLag = 2;     // phase 2 of an item runs kLag iterations after its phase 1
constexpr int kQBufs = 4;   // query / normaliser buffers (items i-2 .. i+1)
constexpr int kMaxLocalItems = 760;  // items per workgroup (their descriptors sit in LDS)
constexpr int kMaxSpins = 1 << 16;     // polls of another workgroup's value (about 1 us each)
constexpr int kMaxProbs = 4096;        // problems the descriptor builder scans in LDS
constexpr unsigned kPending = 0x7FC0DEADu;  // NaN pattern: value not published yet

// One item: (unit = p * h_kv + g, chunk index within the unit, L_p, stat_base) with
// stat_base = tok_off[p] * h_kv + g * L_p, the element offset of the unit's mu / sigma row (the
// unit's keys start at element stat_base * d).  stat_base < 2^31 is checked at launch.
typedef int4 ItemDesc;

struct PipeArgs {
  const uint16_t* q_win;
  const uint16_t* k;
  const ItemDesc* desc;  // [total_items]
  int G;                 // query heads per kv head
  float c;               // softmax scale * log2(e)
  float* row_max;
  float* row_sum;
  float* mu;
  float* sigma;
  float2* part;  // [n_units][max_items][ROWS]
  float* fin;    // [n_units][ROWS]
  int* status;
  int max_items;
  int total_items;
};

struct Item {
  int unit, c, L, n, sbase;  // n = items of the unit
};

__device__ __forceinline__ int sread(int x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ __forceinline__ Item unpack(const ItemDesc& d) {
  Item it;
  it.unit = sread(d.x);
  it.c = sread(d.y);
  it.L = sread(d.z);
  it.sbase = sread(d.w);
  it.n = (it.L + kItemKeys - 1) / kItemKeys;
  return it;
}

__device__ __forceinline__ float sum_halves(float x) {  // x + x of lane ^ 32
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float max_halves(float x) {  // max(x, x of lane ^ 32)
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Device-scope accesses for values exchanged between workgroups.
__device__ __forceinline__ void put_u64(void* p, unsigned long long v) {
  __hip_atomic_store(reinterpret_cast<unsigned long long*>(p), v, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long get_u64(const void* p) {
  return __hip_atomic_load(reinterpret_cast<const unsigned long long*>(p), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void put_u32(void* p, unsigned v) {
  __hip_atomic_store(reinterpret_cast<unsigned*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned get_u32(const void* p) {
  return __hip_atomic_load(reinterpret_cast<const unsigned*>(p), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

// Merge (m2, z2) into (m, z); base-2 units, z relative to 2^m, m = -inf for "no key".
__device__ __forceinline__ void merge_into(float& m, float& z, float m2, float z2) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) return;
  const float a = (m == -INFINITY) ? 0.f : z * __builtin_amdgcn_exp2f(m - mn);
  const float b = (m2 == -INFINITY) ? 0.f : z2 * __builtin_amdgcn_exp2f(m2 - mn);
  m = mn;
  z = a + b;
}

template <int D, int NB> struct Geo {
  static constexpr int R = NB * 32;         // window rows of a unit (G heads x 32)
  static constexpr int NS = D / 16;         // MFMA K steps
  static constexpr int CH = D * 2 / 16;     // 16-byte chunks of a query row
  static constexpr int QELEMS = R * D;      // bf16 elements of one query buffer
  static constexpr int QCHUNKS = R * CH;
  static constexpr int QPT = (QCHUNKS + kThreads - 1) / kThreads;  // staging loads per thread
  static constexpr int RPL = (R + 63) / 64;  // window rows per lane when a wave covers all rows
  // 16-byte chunk `ch` of query row `row` sits at chunk ch ^ (row % CH) of the row in LDS, so that
  // a fragment read of 16 consecutive rows touches 16 different chunks (all banks).
  __device__ static int qslot(int row, int ch) { return row * CH + (ch ^ (row % CH)); }
};

template <int D, int NB>
__global__ __launch_bounds__(kThreads, 1) void window_mu_sigma_fused_kernel(PipeArgs a) {
  using Gm = Geo<D, NB>;
  constexpr int R = Gm::R, NS = Gm::NS, CH = Gm::CH, QPT = Gm::QPT;
  constexpr int RPL = Gm::RPL;
  __shared__ __align__(16) uint16_t qbuf[kQBufs][Gm::QELEMS];
  __shared__ __align__(16) float2 red[2][kWaves][R];  // per-wave (m, z) of the last two items
  __shared__ __align__(16) float bsw[kWaves][R];      // each wave's copy of its phase-2 normalisers
  __shared__ __align__(16) ItemDesc dsh[kMaxLocalItems];  // this workgroup's items, in order
  __shared__ int rcnt;  // phase-1 arrivals: the wave that raises it to 8 (n + 1) is item n's last
  __shared__ int s_fail;  // a wait timed out: every later wait is skipped, outputs become NaN

  const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
  const int wave = sread(threadIdx.x >> 6);
  const int grid = gridDim.x, wg = blockIdx.x;
  const int n_local = wg < a.total_items ? (a.total_items - wg + grid - 1) / grid : 0;
  const float inv_g = 1.f / (float)a.G;
  const float c = a.c;
  if (n_local == 0) return;
  if (threadIdx.x == 0) s_fail = 0;
  auto failed = [&]() {
    return __hip_atomic_load(&s_fail, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) != 0;
  };
  auto fail = [&](int bit) {
    __hip_atomic_store(&s_fail, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    atomicOr(a.status, bit);
  };
  auto exists = [&](int n) { return n >= 0 && n < n_local; };
  auto item_of = [&](int n) { return unpack(dsh[n]); };

  bf16x8_t slot[kSlots][NS];
  bf16x8_t qst[QPT];
  float bq[RPL];  // this lane's polled normalisers, rows lane + 64 k (kept in registers throughout)
#pragma unroll
  for (int k = 0; k < RPL; ++k) bq[k] = 0.f;
  unsigned long long pm[2] = {0ull, 0ull};  // partials requested for the next merge
  float out_val = 0.f;  // this lane's mu (lanes 0-31) or sigma (lanes 32-63) of the last phase 2
  int out_idx = -1;     // its element index, -1 for none

  // ---- loads ---------------------------------------------------------------------------------
  // keys of this wave's tile of an item: a wave-uniform base and this lane's offset (its key
  // clamped into the unit; the lane half selects the 8 elements of each K step)
  auto load_keys = [&](bf16x8_t (&t)[NS], const uint16_t* base, int off) {
#pragma unroll
    for (int s = 0; s < NS; ++s) t[s] = *reinterpret_cast<const bf16x8_t*>(base + off + 16 * s);
  };
  auto load_item_keys = [&](bf16x8_t (&t)[NS], int n) {
    if (exists(n)) {
      const Item it = item_of(n);
      const int t0 = it.c * kItemKeys + wave * 32;
      load_keys(t, a.k + (size_t)(it.sbase + t0) * D, min(l32, it.L - 1 - t0) * D + 8 * half);
    } else {
      load_keys(t, a.k, 8 * half);  // keeps the number of loads per iteration fixed
    }
  };
  // the unit's query rows are contiguous (heads g G .. g G + G - 1 of problem p)
  auto load_queries = [&](int n) {
    const uint16_t* qg = a.q_win + (size_t)(exists(n) ? item_of(n).unit : 0) * R * D;
#pragma unroll
    for (int j = 0; j < QPT; ++j) {
      const int ch = min((int)threadIdx.x + j * kThreads, Gm::QCHUNKS - 1);
      qst[j] = *reinterpret_cast<const bf16x8_t*>(qg + 8 * ch);
    }
  };
  auto store_queries = [&](uint16_t* qb) {
#pragma unroll
    for (int j = 0; j < QPT; ++j) {
      const int ch = threadIdx.x + j * kThreads;
      if (ch < Gm::QCHUNKS)
        *reinterpret_cast<bf16x8_t*>(qb + Gm::qslot(ch / CH, ch % CH) * 8) = qst[j];
    }
  };
  // query fragments of head b (window rows b*32 + l32), all K steps
  auto read_q = [&](bf16x8_t (&qf)[NS], const uint16_t* qb, int b) {
    const int row = b * 32 + l32;
#pragma unroll
    for (int s = 0; s < NS; ++s)
      qf[s] = *reinterpret_cast<const bf16x8_t*>(qb + Gm::qslot(row, 2 * s + half) * 8);
  };

  // ---- phase 1: logits (keys as M), per-wave row maximum and sum -> red[wave] ----------------
  auto phase1 = [&](const bf16x8_t (&t)[NS], const uint16_t* qb, const Item& it, int buf) {
    const int t0 = it.c * kItemKeys + wave * 32;
    const bool edge = t0 + 31 > it.L - 32;
    // window row l32 sees keys <= min(L - 1, L - 32 + l32); the key of register j is
    // t0 + acc_row(j, lane) = t0 + 4 half + 8 (j / 4) + (j % 4)
    const int thr = min(it.L - 1, it.L - 32 + l32) - t0 - 4 * half;
    bf16x8_t qf[NS];
    read_q(qf, qb, 0);
#pragma unroll 1
    for (int b = 0; b < NB; ++b) {
      f32x16_t d = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) d = mfma_step(t[s], qf[s], d);
      if (b + 1 < NB) read_q(qf, qb, b + 1);  // the next head's fragments arrive meanwhile
      if (edge) {
#pragma unroll
        for (int j = 0; j < 16; ++j)
          if (8 * (j >> 2) + (j & 3) > thr) d[j] = -INFINITY;
      }
      float mx[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) mx[u] = fmaxf(fmaxf(d[4 * u], d[4 * u + 1]), fmaxf(d[4 * u + 2], d[4 * u + 3]));
      const float m = max_halves(fmaxf(fmaxf(mx[0], mx[1]), fmaxf(mx[2], mx[3])));
      const float ms = (m == -INFINITY) ? 0.f : m * c;
      float zs[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        zs[u] = __builtin_amdgcn_exp2f(fmaf(d[4 * u], c, -ms));
#pragma unroll
        for (int v = 1; v < 4; ++v) zs[u] += __builtin_amdgcn_exp2f(fmaf(d[4 * u + v], c, -ms));
      }
      const float z = sum_halves((zs[0] + zs[1]) + (zs[2] + zs[3]));
      if (half == 0) red[buf][wave][b * 32 + l32] = make_float2(m == -INFINITY ? -INFINITY : ms, z);
    }
  };

  // ---- phase 2: attention from the unit's normalisers (keys as N), mean and dispersion --------
  auto phase2 = [&](const bf16x8_t (&t)[NS], const uint16_t* qb, const float* bs, const Item& it) {
    const int t0 = it.c * kItemKeys + wave * 32;
    const int key = t0 + l32;
    const bool edge = t0 + 31 > it.L - 32;
    // window row r = acc_row(j, lane) = 4 half + 8 (j / 4) + (j % 4) sees the key iff
    // key <= L - 32 + r
    const int thr = key - (it.L - 32) - 4 * half;
    float ab[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) ab[j] = 0.f;
    // the causal mask only cuts into a unit's last tile: the other tiles take the unmasked loop
    auto accumulate = [&](auto masked) {
#pragma unroll 1
      for (int b = 0; b < NB; ++b) {
        f32x16_t d = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        bf16x8_t qf[NS];
        read_q(qf, qb, b);
#pragma unroll
        for (int s = 0; s < NS; ++s) d = mfma_step(qf[s], t[s], d);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          // window rows 8 q + 4 half + 0..3 of query head b
          const float4 bv = *reinterpret_cast<const float4*>(bs + b * 32 + 8 * q + 4 * half);
          const float bb[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int j = 4 * q + u;
            float e = __builtin_amdgcn_exp2f(fmaf(d[j], c, -bb[u]));
            if (decltype(masked)::value && 8 * q + u < thr) e = 0.f;
            ab[j] += e;
          }
        }
      }
    };
    if (edge) accumulate(std::true_type{});
    else accumulate(std::false_type{});
    // ab[j] = G a[r][key] for the window rows r = acc_row(j, lane); the other 16 are in lane ^ 32
    float sp[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) sp[u] = (ab[u] + ab[u + 4]) + (ab[u + 8] + ab[u + 12]);
    const float mean = sum_halves((sp[0] + sp[1]) + (sp[2] + sp[3])) * (inv_g * (1.f / 32.f));
    float vp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const float dl = fmaf(ab[j], inv_g, -mean);
      vp[j & 3] = fmaf(dl, dl, vp[j & 3]);
    }
    const float var = sum_halves((vp[0] + vp[1]) + (vp[2] + vp[3])) * (1.f / 31.f);
    // the store is issued at the end of the iteration, after the loads the next one waits for
    const float bad = failed() ? __builtin_nanf("") : 0.f;  // a timed-out wait poisons the output
    out_val = (half == 0 ? mean : __builtin_amdgcn_sqrtf(var)) + bad;
    out_idx = key < it.L ? it.sbase + key : -1;
  };

  // ---- merge of the rows an item owns (one wave): lane k takes the partials of items k + 64 q;
  //      pm holds the first row's partials of items lane and lane + 64, requested earlier ----------
  auto owns_rows = [&](const Item& it) { return it.c >= it.n - min(min(it.n, R), grid); };
  auto merge_rows = [&](const Item& it, const unsigned long long (&pm)[2]) {
    const int M = min(min(it.n, R), grid);
    const int r0 = it.c - (it.n - M);
#pragma unroll 1
    for (int row = r0; row < R; row += M) {
      const float2* col = a.part + (size_t)it.unit * a.max_items * R + row;
      float m = -INFINITY, z = 0.f;
#pragma unroll 1
      for (int q = 0; q * 64 < it.n; ++q) {
        const int k = q * 64 + lane;
        unsigned long long v;
        if (row == r0 && q < 2) v = q == 0 ? pm[0] : pm[1];
        else v = get_u64(col + (size_t)min(k, it.n - 1) * R);
        if (k < it.n) {
          int spins = 0;
          while ((unsigned)(v & 0xFFFFFFFFu) == kPending && !failed()) {
            if (++spins > kMaxSpins) {
              fail(1);
              break;
            }
            __builtin_amdgcn_s_sleep(2);
            v = get_u64(col + (size_t)k * R);
          }
          const float2 f = __builtin_bit_cast(float2, v);
          merge_into(m, z, f.x, f.y);
        }
      }
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) merge_into(m, z, __shfl_xor(m, off), __shfl_xor(z, off));
      if (lane == 0) {
        const size_t ri = (size_t)it.unit * R + row;  // = (p h_q + g G + head) * 32 + r
        put_u32(a.fin + ri, __float_as_uint(m + __builtin_log2f(z)));
        a.row_max[ri] = m * kLn2;
        a.row_sum[ri] = z;
      }
    }
  };

  // ---- the item's partial of one row over the waves, max first then the rescaled sum ----------
  auto item_partial = [&](int buf, int row, float& m, float& z) {
    float2 v[kWaves];
#pragma unroll
    for (int w = 0; w < kWaves; ++w) v[w] = red[buf][w][row];
    m = v[0].x;
#pragma unroll
    for (int w = 1; w < kWaves; ++w) m = fmaxf(m, v[w].x);
    z = 0.f;
    if (m != -INFINITY) {
#pragma unroll
      for (int w = 0; w < kWaves; ++w) z = fmaf(v[w].y, __builtin_amdgcn_exp2f(v[w].x - m), z);
    }
  };

  // ---- prologue: item descriptors, queries of item 0 into LDS, keys of items 0 and 1 ----------
  for (int j = threadIdx.x; j < n_local; j += kThreads) dsh[j] = a.desc[(size_t)wg + (size_t)j * grid];
  if (threadIdx.x == 0) rcnt = 0;
  __syncthreads();
  load_queries(0);
  store_queries(qbuf[0]);
  load_queries(1);
  load_item_keys(slot[0], 0);
  load_item_keys(slot[1], 1);

  auto step = [&](auto sc, int i) {
    constexpr int S1 = decltype(sc)::value;            // slot of item i (phase 1)
    constexpr int S2 = (S1 + kSlots - kLag) % kSlots;  // slot of item i - 2, then of item i + 2
    const int n2 = i - kLag;                           // item of phase 2
    const bool has1 = exists(i), has2 = exists(n2);
    Item it1, it2;
    if (has1) it1 = item_of(i);
    if (has2) it2 = item_of(n2);

    // (a) once every wave has finished iteration i - 1, the queries of item i (stored there) are
    //     complete and the buffer of item i + 1 (last read by item i - 3) and red[i & 1] (last read
    //     for item i - 2) are free: store the queries of item i + 1, then phase 1 of item i
    __syncthreads();
    if (exists(i + 1)) store_queries(qbuf[(i + 1) % kQBufs]);
    if (has1) phase1(slot[S1], qbuf[i % kQBufs], it1, i & 1);

    // (b) the last wave to finish phase 1 of item i forms the item's partial of every row and
    //     publishes it for its unit; the others go on at once
    if (has1) {
      int old = 0;
      if (lane == 0)
        old = __hip_atomic_fetch_add(&rcnt, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_WORKGROUP);
      old = sread(old);
      if (old == kWaves * i + kWaves - 1) {
#pragma unroll
        for (int k = 0; k < RPL; ++k) {
          const int row = lane + 64 * k;
          if (row < R) {
            float m, z;
            item_partial(i & 1, row, m, z);
            float2* dst = a.part + ((size_t)it1.unit * a.max_items + it1.c) * R + row;
            put_u64(dst, __builtin_bit_cast(unsigned long long, make_float2(m, z)));
          }
        }
      }
    }

    // (b') the rows item i - 1 owns, merged by one wave (rotating with the iteration)
    if (exists(i - 1) && wave == ((i - 1) & (kWaves - 1))) {
      const Item itm = item_of(i - 1);
      if (owns_rows(itm)) merge_rows(itm, pm);
    }

    // (c) item i - 2's normalisers (requested in the previous iteration) into this wave's LDS
    //     row, then phase 2 of item i - 2
    if (has2) {
#pragma unroll
      for (int k = 0; k < RPL; ++k) {
        const int row = lane + 64 * k;
        if (row < R) {
          int spins = 0;
          while (__float_as_uint(bq[k]) == kPending && !failed()) {
            if (++spins > kMaxSpins) {
              fail(2);
              break;
            }
            __builtin_amdgcn_s_sleep(2);
            bq[k] = __uint_as_float(get_u32(a.fin + (size_t)it2.unit * R + row));
          }
          bsw[wave][row] = bq[k];
        }
      }
      phase2(slot[S2], qbuf[n2 % kQBufs], bsw[wave], it2);
    }

    // (d) the queries of item i + 2, the first partials of item i's next merge, item i - 1's
    //     normalisers, then the keys of item i + 2 into the released slot.  Vector memory
    //     operations of a wave complete in order: what is waited for sooner is requested first,
    //     and this iteration's output store goes last.  Every load is issued unconditionally
    //     (clamped addresses) so that every iteration issues the same number of them and the
    //     waits before phase 1 only cover the keys of the item they need.
    load_queries(i + 2);
    {
      const Item itp = item_of(exists(i) ? i : 0);
      const int M = min(min(itp.n, R), grid);
      const int r0 = max(0, itp.c - (itp.n - M));
      const float2* col = a.part + (size_t)itp.unit * a.max_items * R + r0;
      pm[0] = get_u64(col + (size_t)min(lane, itp.n - 1) * R);
      pm[1] = get_u64(col + (size_t)min(lane + 64, itp.n - 1) * R);
      const Item itf = item_of(exists(i - 1) ? i - 1 : 0);
#pragma unroll
      for (int k = 0; k < RPL; ++k)
        bq[k] = __uint_as_float(get_u32(a.fin + (size_t)itf.unit * R + min(lane + 64 * k, R - 1)));
    }
    load_item_keys(slot[S2], i + 2);
    if (out_idx >= 0) (half == 0 ? a.mu : a.sigma)[out_idx] = out_val;
    out_idx = -1;
  };

  for (int i0 = 0; i0 < n_local + kLag; i0 += kSlots) {
    step(std::integral_constant<int, 0>{}, i0 + 0);
    step(std::integral_constant<int, 1>{}, i0 + 1);
    step(std::integral_constant<int, 2>{}, i0 + 2);
    step(std::integral_constant<int, 3>{}, i0 + 3);
  }
}

// Item descriptors, sentinel-initialised partials and normalisers, cleared status.  Every block
// scans the per-problem item counts itself (n_prob <= kMaxProbs).
__global__ __launch_bounds__(256) void fused_init_kernel(const int32_t* __restrict__ lens,
                                                         const int64_t* __restrict__ tok_off,
                                                         int n_prob, int h_kv, int total_items,
                                                         int max_items, int rows, ItemDesc* desc,
                                                         unsigned* part, unsigned* fin, int* status) {
  __shared__ int pre[kMaxProbs + 1];
  __shared__ int wsum[4];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  // exclusive prefix of h_kv * ceil(L_p / kItemKeys) over the problems
  int carry = 0;
  for (int base = 0; base < n_prob; base += 256) {
    const int p = base + threadIdx.x;
    const int v = p < n_prob ? h_kv * ((lens[p] + kItemKeys - 1) / kItemKeys) : 0;
    int x = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int y = __shfl_up(x, off, 64);
      if (lane >= off) x += y;
    }
    if (lane == 63) wsum[w] = x;
    __syncthreads();
    int before = carry;
    for (int q = 0; q < w; ++q) before += wsum[q];
    if (p < n_prob) pre[p] = before + x - v;
    const int total = carry + wsum[0] + wsum[1] + wsum[2] + wsum[3];
    __syncthreads();
    carry = total;
  }
  if (threadIdx.x == 0) pre[n_prob] = carry;
  __syncthreads();
  const int tid = blockIdx.x * blockDim.x + threadIdx.x, nthr = gridDim.x * blockDim.x;
  for (int q = tid; q < total_items; q += nthr) {
    int lo = 0, hi = n_prob;  // largest p with pre[p] <= q
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (pre[mid] <= q) lo = mid;
      else hi = mid;
    }
    const int L = lens[lo];
    const int nip = (L + kItemKeys - 1) / kItemKeys;
    const int local = q - pre[lo];
    const int g = local / nip, ci = local % nip;
    const long long sbase = (long long)tok_off[lo] * h_kv + (long long)g * L;
    desc[q] = make_int4(lo * h_kv + g, ci, L, (int)sbase);
  }
  const int n_units = n_prob * h_kv;
  const size_t n_part = (size_t)n_units * max_items * rows;  // float2 entries; mark the m word
  for (size_t e = tid; e < n_part; e += nthr) part[2 * e] = kPending;
  for (int e = tid; e < n_units * rows; e += nthr) fin[e] = kPending;
  if (tid == 0) status[0] = 0;
}

}  // namespace

// ------------------------------------------------------------------------------------------------
size_t fused_ws_bytes(const Shape& s) {
  const size_t n_units = (size_t)s.n_prob * s.h_kv;
  const size_t rows = (size_t)s.group() * 32;
  const size_t max_items = (s.max_len + kItemKeys - 1) / kItemKeys;
  size_t b = n_units * max_items * sizeof(ItemDesc);  // bounds the number of items
  b += n_units * max_items * rows * sizeof(float2);
  b += n_units * rows * sizeof(float);
  b += 256;
  return b;
}

bool fused_shape_ok(const Shape& s, float scale) {
  const int G = s.group();
  return s.dtype == kDtBf16 && s.w == 32 && (s.d == 64 || s.d == 128) && (G == 1 || G == 2 || G == 4) &&
         scale > 0.f && s.n_prob <= kMaxProbs;
}

namespace {
int g_resident[64] = {0};  // co-resident workgroups of the fused kernel per device and shape

template <int D, int NB>
hipError_t fused_dispatch(const PipeArgs& base, int total_items, bool* used, hipStream_t st) {
  auto kern = window_mu_sigma_fused_kernel<D, NB>;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const int key = ((dev & 7) << 3) | ((D == 128) << 2) | (NB == 4 ? 2 : (NB == 2 ? 1 : 0));
  int& res = g_resident[key & 63];
  if (res == 0) {
    int per_cu = 0, cus = 0;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(kern),
                                                     kThreads, 0);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    res = per_cu * cus;
  }
  const int grid = min(total_items, res);
  // a unit may have at most one item per workgroup (the deadlock argument above), and a
  // workgroup's item descriptors must fit in LDS
  if (grid <= 0 || base.max_items > grid || (total_items + grid - 1) / grid > kMaxLocalItems) {
    *used = false;
    return hipSuccess;
  }
  PipeArgs args = base;
  args.total_items = total_items;
  void* params[] = {&args};
  e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(kern), dim3(grid), dim3(kThreads),
                                 params, 0, st);
  *used = (e == hipSuccess);
  return e;
}
}  // namespace

hipError_t launch_window_mu_sigma_fused(const Shape& s, const void* q_win, const void* k,
                                        float scale, int total_items, int64_t stat_elems, void* ws,
                                        float* row_max, float* row_sum, float* mu, float* sigma,
                                        bool* used, hipStream_t stream) {
  *used = false;
  if (!fused_shape_ok(s, scale) || stat_elems >= INT32_MAX) return hipSuccess;
  const int n_units = s.n_prob * s.h_kv;
  const int rows = s.group() * 32;
  const int max_items = (s.max_len + kItemKeys - 1) / kItemKeys;
  char* p = static_cast<char*>(ws);
  PipeArgs a;
  ItemDesc* desc = reinterpret_cast<ItemDesc*>(p);
  a.desc = desc;
  p += (size_t)n_units * max_items * sizeof(ItemDesc);
  a.part = reinterpret_cast<float2*>(p);
  p += (size_t)n_units * max_items * rows * sizeof(float2);
  a.fin = reinterpret_cast<float*>(p);
  p += (size_t)n_units * rows * sizeof(float);
  a.status = reinterpret_cast<int*>(p);
  a.q_win = static_cast<const uint16_t*>(q_win);
  a.k = static_cast<const uint16_t*>(k);
  a.G = s.group();
  a.c = scale * kLog2e;
  a.row_max = row_max;
  a.row_sum = row_sum;
  a.mu = mu;
  a.sigma = sigma;
  a.max_items = max_items;
  a.total_items = total_items;
  fused_init_kernel<<<512, 256, 0, stream>>>(s.lens, s.tok_off, s.n_prob, s.h_kv, total_items,
                                             max_items, rows, desc,
                                             reinterpret_cast<unsigned*>(a.part),
                                             reinterpret_cast<unsigned*>(a.fin), a.status);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int G = s.group();
  if (s.d == 128) {
    if (G == 4) return fused_dispatch<128, 4>(a, total_items, used, stream);
    if (G == 2) return fused_dispatch<128, 2>(a, total_items, used, stream);
    return fused_dispatch<128, 1>(a, total_items, used, stream);
  }
  if (G == 4) return fused_dispatch<64, 4>(a, total_items, used, stream);
  if (G == 2) return fused_dispatch<64, 2>(a, total_items, used, stream);
  return fused_dispatch<64, 1>(a, total_items, used, stream);
}

}  // namespace kv
