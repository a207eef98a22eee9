// Single-pass window statistics: row softmax statistics and per-token mean / dispersion
// (section 3.1, Eq. (1), Eq. (3)) reading every cached key once, for bf16 caches with w = 32.
//
// The row normaliser of a window query needs every key of its (problem, kv head) "unit" before any
// token's attention can be formed.  Instead of a second pass over K, each work item keeps its logits
// in registers while the units' statistics are combined across workgroups:
//
//   work item = (unit, chunk of 512 keys); 16 waves x one MFMA tile of 32 keys; rows = G*32 window
//   rows of the kv group (row block b = query head b of the group, row = window position r);
//   1. logits D[key][row] = K Q^T with v_mfma_f32_32x32x16_bf16, keys as the M dimension so that a
//      lane holds one window row and 16 keys (queries from LDS, keys straight from HBM into operand
//      registers; the next item's queries are requested into the other LDS buffer right after the
//      MFMAs, its keys right after this item's partials are published, so both stream in during
//      the unit barrier and the final reduction);
//   2. workgroup row maximum m and, after e = 2^(t - m) in place, row sum z: in-lane over 16 keys,
//      one permlane32 swap for the other 16, then across waves in LDS; (m, z) is published to the
//      unit's partial slot with a write-through store;
//   3. unit barrier: the last workgroup of a unit to publish its partial merges all of them into
//      b = M + log2 Z per row (and the row_max / row_sum outputs) and raises the unit's flag; the
//      others poll the flag.  Exchanged data uses system-scope (write-through, cache-bypassing)
//      accesses ordered by s_waitcnt, so no L2 write-back or invalidation is needed; the grid is
//      launched cooperatively so every workgroup is resident, and a unit spans at most one grid;
//   4. a = e * 2^(m - b) / G summed over the group's heads gives the window row means a[r] of the
//      lane's 16 keys; a per-wave 32 x 32 LDS transpose gives each lane one key and 16 rows, so the
//      mean over r and the two-pass sample variance are in-lane plus one permlane32 swap.
//
// Work items are dealt round-robin (item i -> workgroup i % grid), units in order, so a unit's
// items are resident together and the barrier cannot deadlock.  Every wait is bounded.
#include "common.h"
#include "kernels.h"

namespace kv {

namespace {

constexpr int kWaves = 16;
constexpr int kThreads = kWaves * 64;
constexpr int kTiles = 1;
constexpr int kMaxSpins = 1 << 22;
constexpr unsigned kFinPending = 0x7FC0DEADu;  // NaN pattern: final row value not published yet

struct FusedArgs {
  const uint16_t* q_win;
  const uint16_t* k;
  const int32_t* lens;
  const int64_t* tok_off;
  int n_prob, h_q, h_kv;
  float c;  // softmax scale * log2(e)
  float* row_max;
  float* row_sum;
  float* mu;
  float* sigma;
  float2* part;       // [n_units][max_chunks][ROWS]
  float* fin;         // [n_units][ROWS]
  int* cnt;           // [n_units]
  int* flag;          // [n_units]
  int* item_prefix;   // [n_prob + 1]
  int* status;        // [1]
  int max_chunks;
  int total_items;
};

__device__ __forceinline__ float sum_halves(float x) {  // x + x of lane ^ 32
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float max_halves(float x) {  // max(x, x of lane ^ 32)
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Coherent (write-through / cache-bypassing) accesses for data exchanged between workgroups.
__device__ __forceinline__ void publish_f2(float2* p, float2 v) {
  __hip_atomic_store(reinterpret_cast<unsigned long long*>(p), __builtin_bit_cast(unsigned long long, v),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}
__device__ __forceinline__ float2 fetch_f2(const float2* p) {
  return __builtin_bit_cast(float2, __hip_atomic_load(reinterpret_cast<const unsigned long long*>(p),
                                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM));
}
__device__ __forceinline__ void publish_f(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}
__device__ __forceinline__ float fetch_f(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

struct Item {
  int p, g, c, L, nch, unit;
};

__device__ __forceinline__ Item decode_item(const FusedArgs& a, int item) {
  // problem: largest p with item_prefix[p] <= item
  int lo = 0, hi = a.n_prob;  // item_prefix[0] = 0 <= item < item_prefix[n_prob]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (a.item_prefix[mid] <= item) lo = mid;
    else hi = mid;
  }
  // every field is the same for the whole workgroup: keep them in scalar registers
  Item it;
  it.p = __builtin_amdgcn_readfirstlane(lo);
  it.L = __builtin_amdgcn_readfirstlane(a.lens[it.p]);
  it.nch = (it.L + kFusedChunk - 1) / kFusedChunk;
  const int local = __builtin_amdgcn_readfirstlane(item - a.item_prefix[it.p]);
  it.g = local / it.nch;
  it.c = local % it.nch;
  it.unit = it.p * a.h_kv + it.g;
  return it;
}

// Query rows of one unit in LDS: row pitch CHUNKS + 1 sixteen-byte slots (the pad slot shifts
// consecutive rows by four banks, so a fragment read of 16 rows is conflict-free and every K-step
// offset is an immediate).  Filled by direct-to-LDS loads, one contiguous kilobyte per wave
// instruction; a lane whose slot is a pad loads its row's first chunk again.
template <int D> struct QPitch {
  static constexpr int CHUNKS = D * 2 / 16;
  static constexpr int SLOTS = CHUNKS + 1;
};

// Issued by waves first_wave .. kWaves-1 only.
template <int D, int NB>
__device__ __forceinline__ void request_queries(const FusedArgs& a, const Item& it, uint16_t* qbuf,
                                                int first_wave) {
  constexpr int CHUNKS = QPitch<D>::CHUNKS, SLOTS = QPitch<D>::SLOTS;
  constexpr int ROWS = NB * 32;
  constexpr int PER_WAVE_INSTR = 64;  // 16-byte slots per wave instruction
  constexpr int N_INSTR = (ROWS * SLOTS + PER_WAVE_INSTR - 1) / PER_WAVE_INSTR;
  const int G = a.h_q / a.h_kv;
  const uint16_t* qg = a.q_win + ((size_t)it.p * a.h_q + (size_t)it.g * G) * 32 * D;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int gi = wave - first_wave; gi >= 0 && gi < N_INSTR; gi += kWaves - first_wave) {
    const int slot_lin = gi * PER_WAVE_INSTR + lane;  // LDS 16-byte slot written by this lane
    int m = slot_lin / SLOTS, q = slot_lin % SLOTS;
    if (q == CHUNKS) q = 0;               // pad slot
    if (m >= ROWS) m = ROWS - 1, q = 0;   // beyond the last row (inside the buffer's tail)
    __builtin_amdgcn_global_load_lds(qg + (size_t)m * D + q * 8, qbuf + gi * PER_WAVE_INSTR * 8,
                                     16, 0, 0);
  }
}

}  // namespace

template <int D, int NB>
__global__ __launch_bounds__(kThreads, 1) void window_mu_sigma_fused_kernel(FusedArgs a) {
  constexpr int ROWS = NB * 32;
  constexpr int SLOTS = QPitch<D>::SLOTS;
  constexpr int QBUF = ((ROWS * SLOTS + 63) / 64) * 64 * 8;  // elements, whole wave instructions
  constexpr int NS = D / 16;                                 // MFMA K steps
  constexpr int PARTS = kThreads / ROWS;                     // slices of a unit's chunks
  constexpr int TP = 33;                                     // transpose tile pitch (floats)
  __shared__ __align__(16) uint16_t qbuf[2][QBUF];
  __shared__ __align__(16) float red[kWaves][ROWS];
  __shared__ __align__(16) float srow[ROWS];  // workgroup row max, then 2^(m - b) / G
  // per-wave 32x32 transpose tiles of the finalisation; the last workgroup's merge reuses them
  __shared__ __align__(16) float xt[kWaves * 32 * TP];
  static_assert(kWaves * 32 * TP >= 2 * PARTS * ROWS, "merge scratch must fit in the tiles");
  __shared__ int s_last;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5, l32 = lane & 31;
  const int G = a.h_q / a.h_kv;
  const float inv_g = 1.f / (float)G;

  int item = blockIdx.x;
  if (item >= a.total_items) return;
  Item it = decode_item(a, item);
  Frags<kDtBf16, D> kf;
  auto key_row = [&](const Item& x) {
    const int64_t off = (int64_t)__builtin_amdgcn_readfirstlane((int)(a.tok_off[x.p] & 0xFFFFFFFF)) |
                        ((int64_t)__builtin_amdgcn_readfirstlane((int)(a.tok_off[x.p] >> 32)) << 32);
    const uint16_t* kg = a.k + ((size_t)off * a.h_kv + (size_t)x.g * x.L) * D;
    const int key = min(x.c * kFusedChunk + wave * 32 + l32, x.L - 1);
    return kg + (size_t)key * D;
  };
  request_queries<D, NB>(a, it, qbuf[0], 0);
  kf.load_global(key_row(it), half);

  for (int iter = 0; item < a.total_items; ++iter, item += gridDim.x) {
    const int nxt = item + gridDim.x;
    const bool has_next = nxt < a.total_items;
    const Item nx = has_next ? decode_item(a, nxt) : it;
    const uint16_t* qb = qbuf[iter & 1];
    __builtin_amdgcn_s_waitcnt(0);  // this item's queries (direct-to-LDS) and keys have landed
    __syncthreads();

    // ---- 1. logits D[key][row]: lane = window row b*32 + (lane % 32), 16 keys per lane ----------
    f32x16_t acc[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      f32x16_t d = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      const uint16_t* qrow = qb + ((b * 32 + l32) * SLOTS + half) * 8;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const bf16x8_t qa = *reinterpret_cast<const bf16x8_t*>(qrow + 16 * s);
        d = mfma_step(kf.v[s], qa, d);
      }
      acc[b] = d;
    }

    // ---- causal / ragged mask: row r = lane % 32 sees keys <= L - 32 + r -----------------------
    const int t0 = it.c * kFusedChunk + wave * 32;
    if (t0 + 31 > it.L - 32) {
      const int lim = min(it.L - 1, it.L - 32 + l32);
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int j = 0; j < 16; ++j)
          if (t0 + acc_row(j, lane) > lim) acc[b][j] = -INFINITY;
    }

    // ---- 2a. workgroup row maximum (in-lane over 16 keys, the other 16 in lane ^ 32) ----------
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      float m = acc[b][0];
#pragma unroll
      for (int j = 1; j < 16; ++j) m = fmaxf(m, acc[b][j]);
      m = max_halves(m);
      if (half == 0) red[wave][b * 32 + l32] = m;
    }
    __syncthreads();
    if (threadIdx.x < ROWS) {
      float m = red[0][threadIdx.x];
#pragma unroll
      for (int w = 1; w < kWaves; ++w) m = fmaxf(m, red[w][threadIdx.x]);
      srow[threadIdx.x] = m * a.c;  // in base-2 logit units (c > 0)
    }
    __syncthreads();

    // ---- 2b. e = 2^(t - m) in place and workgroup row sum ------------------------------------
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const float mm = srow[b * 32 + l32];
      float z = 0.f;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float e = __builtin_amdgcn_exp2f(fmaf(acc[b][j], a.c, -mm));
        acc[b][j] = e;
        z += e;
      }
      z = sum_halves(z);
      if (half == 0) red[wave][b * 32 + l32] = z;
    }
    __syncthreads();
    const size_t ubase = (size_t)it.unit * a.max_chunks * ROWS;
    if (threadIdx.x < ROWS) {
      float z = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) z += red[w][threadIdx.x];
      publish_f2(a.part + ubase + (size_t)it.c * ROWS + threadIdx.x, make_float2(srow[threadIdx.x], z));
      __builtin_amdgcn_s_waitcnt(0);  // the partial has reached memory before the counter moves
    }
    __syncthreads();

    // ---- 3. unit barrier ------------------------------------------------------------------------
    if (threadIdx.x == 0) {
      const int old = __hip_atomic_fetch_add(&a.cnt[it.unit], 1, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT);
      s_last = (old == it.nch - 1);
    }
    __syncthreads();
    // The next item's queries and keys stream in while this unit's statistics are combined and
    // finalised.  They are issued after the publish (so that its wait covers only the partial
    // store), and the waves that poll for the unit's final values issue theirs only after the
    // poll: vector loads of a wave complete in order, so a poll behind a prefetch would wait for it.
    constexpr int kPollWaves = (ROWS + 63) / 64;
    if (has_next && wave >= kPollWaves) {
      request_queries<D, NB>(a, nx, qbuf[(iter + 1) & 1], kPollWaves);
      kf.load_global(key_row(nx), half);
    }
    if (s_last) {
      // merge every partial of the unit: PARTS slices per row, loads issued in batches of 8
      float2* comb = reinterpret_cast<float2*>(xt);
      const int row = threadIdx.x % ROWS, part = threadIdx.x / ROWS;
      float M = -INFINITY, Z = 0.f;
      for (int ch0 = part; ch0 < it.nch; ch0 += 8 * PARTS) {
        float2 o[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int ch = ch0 + q * PARTS;
          o[q] = ch < it.nch ? fetch_f2(a.part + ubase + (size_t)ch * ROWS + row)
                             : make_float2(-INFINITY, 0.f);
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) merge_mz(M, Z, o[q].x, o[q].y);
      }
      comb[part * ROWS + row] = make_float2(M, Z);
      __syncthreads();
      if (threadIdx.x < ROWS) {
        float2 r = comb[threadIdx.x];
#pragma unroll
        for (int q = 1; q < PARTS; ++q) merge_mz(r.x, r.y, comb[q * ROWS + threadIdx.x].x, comb[q * ROWS + threadIdx.x].y);
        const float bfin = r.x + log2f(r.y);
        publish_f(a.fin + (size_t)it.unit * ROWS + threadIdx.x, bfin);
        const int hl = threadIdx.x / 32, rr = threadIdx.x % 32;
        const size_t ri = ((size_t)it.p * a.h_q + (size_t)it.g * G + hl) * 32 + rr;
        a.row_max[ri] = r.x * kLn2;
        a.row_sum[ri] = r.y;
        srow[threadIdx.x] = __builtin_amdgcn_exp2f(srow[threadIdx.x] - bfin) * inv_g;
      }
    } else if (threadIdx.x < ROWS) {
      // each row polls its own final value; the init kernel set it to a NaN sentinel
      const float* fp = a.fin + (size_t)it.unit * ROWS + threadIdx.x;
      float bfin = fetch_f(fp);
      int spins = 0;
      while (__float_as_uint(bfin) == kFinPending) {
        if (++spins > kMaxSpins) {
          atomicOr(a.status, 1);
          break;
        }
        __builtin_amdgcn_s_sleep(1);
        bfin = fetch_f(fp);
      }
      srow[threadIdx.x] = __builtin_amdgcn_exp2f(srow[threadIdx.x] - bfin) * inv_g;
    }
    if (has_next && wave < kPollWaves) kf.load_global(key_row(nx), half);
    __syncthreads();

    // ---- 4. group mean over heads, then mean and dispersion over the window --------------------
    float abar[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) abar[j] = 0.f;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const float al = srow[b * 32 + l32];
#pragma unroll
      for (int j = 0; j < 16; ++j) abar[j] = fmaf(acc[b][j], al, abar[j]);
    }
    // transpose through LDS: tile[key][r], this lane holds r = lane % 32 of keys acc_row(j, lane)
    float* tile = xt + wave * 32 * TP;
#pragma unroll
    for (int j = 0; j < 16; ++j) tile[acc_row(j, lane) * TP + l32] = abar[j];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    float v[16];
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      v[i] = tile[l32 * TP + 16 * half + i];  // key l32, rows 16 half .. 16 half + 15
      s += v[i];
    }
    const float mean = sum_halves(s) * (1.f / 32.f);
    float var = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float dl = v[i] - mean;
      var = fmaf(dl, dl, var);
    }
    var = sum_halves(var) * (1.f / 31.f);
    const int64_t toff = (int64_t)__builtin_amdgcn_readfirstlane((int)(a.tok_off[it.p] & 0xFFFFFFFF)) |
                         ((int64_t)__builtin_amdgcn_readfirstlane((int)(a.tok_off[it.p] >> 32)) << 32);
    const size_t stat_base = (size_t)toff * a.h_kv + (size_t)it.g * it.L;
    const int key = t0 + l32;
    if (key < it.L) {
      if (half == 0) a.mu[stat_base + key] = mean;
      else a.sigma[stat_base + key] = sqrtf(var);
    }
    it = nx;
  }
}

// Zero the unit counters and flags and lay out the work items (exclusive prefix over problems).
__global__ __launch_bounds__(1024) void fused_init_kernel(const int32_t* __restrict__ lens, int n_prob,
                                                          int h_kv, int n_units, int rows, int* cnt,
                                                          unsigned* fin, int* item_prefix, int* status) {
  __shared__ int part[1024];
  for (int u = threadIdx.x; u < n_units; u += blockDim.x) cnt[u] = 0;
  for (int i = threadIdx.x; i < n_units * rows; i += blockDim.x) fin[i] = kFinPending;
  if (threadIdx.x == 0) status[0] = 0;
  const int per = (n_prob + 1023) / 1024;
  const int lo = threadIdx.x * per, hi = min(n_prob, lo + per);
  int s = 0;
  for (int p = lo; p < hi; ++p) s += h_kv * ((lens[p] + kFusedChunk - 1) / kFusedChunk);
  part[threadIdx.x] = s;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const int add = threadIdx.x >= off ? part[threadIdx.x - off] : 0;
    __syncthreads();
    part[threadIdx.x] += add;
    __syncthreads();
  }
  int run = part[threadIdx.x] - s;  // exclusive prefix of this thread's range
  for (int p = lo; p < hi; ++p) {
    item_prefix[p] = run;
    run += h_kv * ((lens[p] + kFusedChunk - 1) / kFusedChunk);
  }
  if (threadIdx.x == 1023) item_prefix[n_prob] = part[1023];
}

// ------------------------------------------------------------------------------------------------
size_t fused_ws_bytes(const Shape& s) {
  const size_t n_units = (size_t)s.n_prob * s.h_kv;
  const size_t rows = (size_t)s.group() * 32;
  const size_t max_chunks = (s.max_len + kFusedChunk - 1) / kFusedChunk;
  size_t b = n_units * max_chunks * rows * sizeof(float2);
  b += n_units * rows * sizeof(float);
  b += 2 * n_units * sizeof(int);
  b += (s.n_prob + 1) * sizeof(int) + sizeof(int);
  return b;
}

bool fused_shape_ok(const Shape& s, float scale) {
  const int G = s.group();
  return s.dtype == kDtBf16 && s.w == 32 && (s.d == 64 || s.d == 128) && (G == 1 || G == 2 || G == 4) &&
         scale > 0.f;
}

namespace {
int g_resident[64] = {0};  // co-resident workgroups of the fused kernel per device and shape

template <int D, int NB>
hipError_t fused_dispatch(const FusedArgs& base, int total_items, bool* used, hipStream_t st) {
  auto kern = window_mu_sigma_fused_kernel<D, NB>;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const int slot = ((dev & 15) << 2) | ((D == 128) << 1) | (NB == 4);
  int& res = g_resident[slot & 63];
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
  if (grid <= 0 || base.max_chunks > grid) {  // every unit must fit in one grid of items
    *used = false;
    return hipSuccess;
  }
  FusedArgs args = base;
  args.total_items = total_items;
  void* params[] = {&args};
  e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(kern), dim3(grid), dim3(kThreads),
                                 params, 0, st);
  *used = (e == hipSuccess);
  return e;
}
}  // namespace

hipError_t launch_window_mu_sigma_fused(const Shape& s, const void* q_win, const void* k,
                                        float scale, int total_items, void* ws, float* row_max,
                                        float* row_sum, float* mu, float* sigma, bool* used,
                                        hipStream_t stream) {
  *used = false;
  if (!fused_shape_ok(s, scale)) return hipSuccess;
  const int n_units = s.n_prob * s.h_kv;
  const int rows = s.group() * 32;
  const int max_chunks = (s.max_len + kFusedChunk - 1) / kFusedChunk;
  char* p = static_cast<char*>(ws);
  FusedArgs a;
  a.part = reinterpret_cast<float2*>(p);
  p += (size_t)n_units * max_chunks * rows * sizeof(float2);
  a.fin = reinterpret_cast<float*>(p);
  p += (size_t)n_units * rows * sizeof(float);
  a.cnt = reinterpret_cast<int*>(p);
  p += (size_t)n_units * sizeof(int);
  a.flag = reinterpret_cast<int*>(p);
  p += (size_t)n_units * sizeof(int);
  a.item_prefix = reinterpret_cast<int*>(p);
  p += (size_t)(s.n_prob + 1) * sizeof(int);
  a.status = reinterpret_cast<int*>(p);
  a.q_win = static_cast<const uint16_t*>(q_win);
  a.k = static_cast<const uint16_t*>(k);
  a.lens = s.lens;
  a.tok_off = s.tok_off;
  a.n_prob = s.n_prob;
  a.h_q = s.h_q;
  a.h_kv = s.h_kv;
  a.c = scale * kLog2e;
  a.row_max = row_max;
  a.row_sum = row_sum;
  a.mu = mu;
  a.sigma = sigma;
  a.max_chunks = max_chunks;
  a.total_items = total_items;
  fused_init_kernel<<<1, 1024, 0, stream>>>(s.lens, s.n_prob, s.h_kv, n_units, rows, a.cnt,
                                            reinterpret_cast<unsigned*>(a.fin), a.item_prefix,
                                            a.status);
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
