// HIGGS encoder (Alg. 1, RHT-VQ, with the grid of Alg. 2) on the GPU.
//
// One wavefront encodes one group of g consecutive weights of one row:
//   s = ||w||_2                      (fp64 sum of squares, fixed reduction tree)
//   w_dag = H (sigma * (w / s))      (fp64, in-register / cross-lane butterflies)
//   code_j = argmin_k ||w_dag[jp:(j+1)p] - G_k||^2, lowest k on ties
//   scale = fp16(s / sqrt(g))        (one rounding from fp64)
// The search compares c_k = |G_k|^2 / 2 - <v, G_k>, which orders the grid
// points exactly as the squared distance does, in fp64. To take the running
// minimum and its index in one v_min_f64, each candidate's value is shifted
// by a power of two S that makes it positive and its 10 lowest mantissa bits
// are replaced by k: positive doubles order as their bit patterns, so the
// minimum is the smallest value, ties (and values within 1024 ulps of S,
// S 2^-42) going to the lowest k. |v| <= sqrt(g) for a p-vector of a rotated
// group (its squared norm sums to g), so |c_k| <= R^2 / 2 + sqrt(g) R with R
// the largest grid-point norm; each block takes S = the least power of two
// >= max(1024, 2 (R^2 / 2 + sqrt(g) R)) from the grid it loads. Every grid of
// unit-variance points gets S = 1024, where the order differs from the plain
// fp64 distance only at squared-distance gaps below ~5e-10; the band is
// S 2^-41 in general, below 1e-6 for grids whose points have norms <= 1024.
// Candidates: with a search index built from the same grid, a p-vector is
// compared with the grid points of its bucket's list only (exact pruning,
// below), which holds every point whose search value can be the least one
// for a vector in that bucket; vectors outside the bucketed square, and every
// vector without a matching index, scan all n points. The chosen code is the
// one a full scan gives.
// Codes are packed LSB-first into the row's bit stream through LDS.

#include <algorithm>
#include <cmath>
#include <type_traits>

#include "internal.h"
#include "wave_fwht.h"

namespace higgs {
namespace {

constexpr int kWaves = 4;
constexpr int kMaxN = 1024;
constexpr int kMaxG = 4096;
constexpr double kMinShift = 1024.0;   // least shift of the search values
constexpr uint32_t kIndexMask = 1023;  // low mantissa bits that carry the index (n <= 1024)

// min(best, c with its 10 lowest mantissa bits replaced by k). c and best
// are positive and finite, so no NaN handling is needed: one bit-field insert
// on the low word and one v_min_f64 (the compiler's fmin would first quieten
// both operands).
__device__ inline double min_indexed(double best, double c, uint32_t k, uint32_t index_mask) {
  const uint64_t u = __builtin_bit_cast(uint64_t, c);
  uint32_t lo;
  // lo = (k & index_mask) | (low word of c & ~index_mask); index_mask in a VGPR
  __asm__("v_bfi_b32 %0, %1, %2, %3" : "=v"(lo) : "v"(index_mask), "s"(k), "v"(uint32_t(u)));
  const double ck = __builtin_bit_cast(double, (u & 0xffffffff00000000ull) | uint64_t(lo));
  double r;
  __asm__("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(best), "v"(ck));
  return r;
}

// fp64 -> IEEE binary16 bits, round to nearest even, for finite x >= 0.
__device__ inline uint16_t f64_to_f16_rne(double x) {
  if (!(x > 0.0)) return 0;
  if (x >= 65520.0) return 0x7C00;                  // rounds to +infinity
  const int e = ilogb(x);                           // x in [2^e, 2^(e+1))
  const int qe = e - 10 > -24 ? e - 10 : -24;       // fp16 spacing in that binade
  const double r = ldexp(rint(ldexp(x, -qe)), qe);  // exact fp16 value
  const _Float16 h = static_cast<_Float16>(static_cast<float>(r));  // exact conversions
  return __builtin_bit_cast(uint16_t, h);
}

template <typename InT>
__device__ inline double to_f64(InT v);
template <>
__device__ inline double to_f64<float>(float v) { return double(v); }
template <>
__device__ inline double to_f64<uint16_t>(uint16_t v) {
  return double(__uint_as_float(uint32_t(v) << 16));
}

template <int E, typename InT>
__device__ inline void load_group(const InT* __restrict__ src, double (&v)[E]) {
  constexpr int kBytes = E * int(sizeof(InT));
  if constexpr (kBytes % 16 == 0) {
    constexpr int kPer = 16 / int(sizeof(InT));
#pragma unroll
    for (int q = 0; q < kBytes / 16; ++q) {
      const u32x4 u = load_stream16(reinterpret_cast<const char*>(src) + 16 * q);
      const InT* e = reinterpret_cast<const InT*>(&u);
#pragma unroll
      for (int i = 0; i < kPer; ++i) v[q * kPer + i] = to_f64<InT>(e[i]);
    }
  } else {
#pragma unroll
    for (int i = 0; i < E; ++i) v[i] = to_f64<InT>(src[i]);
  }
}

// ---------------------------------------------------------------------------
// Search index: exact pruning of the nearest-point search. The square
// [-kBR, kBR)^P is cut into kNB^P buckets. Point k may be left out of bucket
// B's list when some point j is nearer than k to every point of B, by a
// margin m in squared distance: dmin(k, B)^2 > dmax(j, B)^2 + m, with dmin /
// dmax the least and the largest distance from the point to the (slightly
// widened) box of B. Since c_k - c_j = (|v - G_k|^2 - |v - G_j|^2) / 2, such
// a k has a search value above j's by more than m / 2 for every v in B; m
// (2^-30 S, S the search shift of the largest group size, which bounds the
// shift of every group size) is far above the 2^-42 S by which the index
// bits move a value and the rounding of the values, so k is never the least
// one. A list is never empty: it holds the point that sets the bound.
//
// The index is built once per grid (one wavefront per bucket, then one block
// that lays the lists out back to back) and read by every quantize block into
// LDS. It carries a hash of the grid's values, the margin and its geometry;
// a block that loads a grid whose hash differs, or an index that is missing
// or does not fit, scans all n points for every vector, so an index can only
// change the speed of a call, never its codes.
// ---------------------------------------------------------------------------
constexpr double kBR = 4.0;      // half side of the bucketed square
constexpr double kBEps = 1e-9;   // widening of a bucket's box (bucket-index rounding)
constexpr uint32_t kIndexMagic = 0x49534748u;
constexpr int kSlotCap = 64;     // entries per bucket while the index is built
// Buckets per axis: 512 for p = 1; for p = 2, 64 (128 for the 1024-point
// grid, whose lists would average about 9 points at 64: 3 at 128).
__host__ __device__ constexpr int index_nb(int p, int n) {
  return p == 1 ? 512 : (n >= 256 ? 128 : 64);
}
__host__ __device__ constexpr int index_cells(int p, int n) {
  return p == 1 ? index_nb(p, n) : index_nb(p, n) * index_nb(p, n);
}
template <int P, int N>
struct Buckets {
  static constexpr int kNB = index_nb(P, N), kCells = index_cells(P, N);
};

__host__ __device__ constexpr int64_t align16(int64_t b) { return (b + 15) / 16 * 16; }
// list entries a quantize block holds in LDS
__host__ __device__ constexpr int index_list_cap(int p, int n) {
  return p == 1 ? 2048 : (n <= 64 ? 8192 : 32768);
}

struct IndexHeader {
  uint32_t magic, p, n, nb;
  uint32_t total, usable, reserved0, reserved1;
  uint64_t hash;
  double margin, half_side;
  uint64_t reserved;
};
static_assert(sizeof(IndexHeader) == 64, "index header");

// header | u16 offsets [cells + 1] | u16 lists [cap] | build scratch: u16
// counts [cells], u16 slots [cells][kSlotCap]; regions 16-byte aligned
struct IndexLayout {
  int64_t offsets, list, counts, slots, bytes;
};
__host__ __device__ constexpr IndexLayout index_layout(int p, int n) {
  const int64_t cells = index_cells(p, n);
  const int64_t offsets = 64;
  const int64_t list = offsets + align16((cells + 1) * 2);
  const int64_t counts = list + align16(int64_t(index_list_cap(p, n)) * 2);
  const int64_t slots = counts + align16(cells * 2);
  return IndexLayout{offsets, list, counts, slots, slots + cells * kSlotCap * 2};
}

// the search-value shift for groups of g weights: a power of two at least
// twice the largest |c_k| (see the file's header)
__device__ inline double search_shift(double r2, int g) {
  const double bound = 2.0 * (0.5 * r2 + sqrt(double(g)) * sqrt(r2));
  return bound <= kMinShift ? kMinShift : exp2(ceil(log2(bound)));
}

// hash of grid point k (its index and the bits of its coordinates); the
// grid's hash is the sum over its points (mod 2^64)
template <int P>
__device__ inline uint64_t point_hash(const float* c, int k) {
  uint64_t h = splitmix64_at(0x48474753ull, uint64_t(k));
#pragma unroll
  for (int t = 0; t < P; ++t) h = splitmix64_at(h, __float_as_uint(c[t]));
  return h;
}

// dmin^2 and dmax^2 from point g to the box [lo, lo + w]^P (widened by kBEps)
template <int P>
__device__ inline void box_d2(const double* g, const double (&lo)[P], double w, double& dmin2,
                              double& dmax2) {
  dmin2 = 0.0;
  dmax2 = 0.0;
#pragma unroll
  for (int t = 0; t < P; ++t) {
    const double a = lo[t] - kBEps - g[t], b = g[t] - (lo[t] + w + kBEps);
    const double dn = fmax(0.0, fmax(a, b));
    const double dx = fmax(fabs(a), fabs(b));
    dmin2 = fma(dn, dn, dmin2);
    dmax2 = fma(dx, dx, dmax2);
  }
}

// Bucket index along one axis, or -1 outside [-kBR, kBR) (or for NaN).
__device__ inline int bucket_axis(double v, int nb) {
  const double f = floor((v + kBR) * (double(nb) / (2.0 * kBR)));
  return (f >= 0.0 && f < double(nb)) ? int(f) : -1;
}

// In place: counts a[0 .. n) -> exclusive offsets, a[n] = total (n + 1
// entries; block-wide, every thread of the block calls it). Returns the
// total (every thread). s_tmp: one entry per wave.
__device__ inline int block_offsets(uint32_t* a, int n, int tid, int nthreads, uint32_t* s_tmp) {
  const int per = (n + nthreads - 1) / nthreads;
  const int b0 = min(n, tid * per), b1 = min(n, b0 + per);
  uint32_t local = 0;
  for (int i = b0; i < b1; ++i) local += a[i];
  // inclusive scan over the wave
  const int lane = tid & 63, wave = tid >> 6;
  uint32_t inc = local;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t o = uint32_t(__shfl_up(int(inc), d));
    if (lane >= d) inc += o;
  }
  if (lane == 63) s_tmp[wave] = inc;
  __syncthreads();
  uint32_t base = 0, total = 0;
  for (int w = 0; w < nthreads / 64; ++w) {
    if (w < wave) base += s_tmp[w];
    total += s_tmp[w];
  }
  uint32_t run = base + inc - local;
  for (int i = b0; i < b1; ++i) {
    const uint32_t c = a[i];
    a[i] = run;
    run += c;
  }
  if (tid == 0) a[n] = total;
  __syncthreads();
  return int(total);
}

// One wavefront per bucket: the bucket's list into its slot (at most
// kSlotCap entries kept, the full count written).
template <int P, int N>
__global__ __launch_bounds__(256) void index_slots_kernel(const float* __restrict__ grid, int n,
                                                          uint8_t* __restrict__ index) {
  using B = Buckets<P, N>;
  constexpr double kW = 2.0 * kBR / B::kNB;
  const IndexLayout L = index_layout(P, n);
  const int lane = int(threadIdx.x) & 63;
  const int b = int(blockIdx.x) * 4 + (int(threadIdx.x) >> 6);
  if (b >= B::kCells) return;  // whole waves
  double lo[P];
  lo[0] = -kBR + kW * (b % B::kNB);
  if constexpr (P == 2) lo[1] = -kBR + kW * (b / B::kNB);
  // the margin, from the largest squared norm; the bound u = min_j dmax^2
  double r2 = 0.0, u = INFINITY;
  for (int k = lane; k < n; k += 64) {
    double gk[P], h = 0.0;
#pragma unroll
    for (int t = 0; t < P; ++t) {
      gk[t] = double(grid[k * P + t]);
      h += gk[t] * gk[t];
    }
    r2 = fmax(r2, h);
    double dn, dx;
    box_d2<P>(gk, lo, kW, dn, dx);
    u = fmin(u, dx);
  }
  r2 = wave_max(r2, lane);
  u = -wave_max(-u, lane);
  const double m = ldexp(search_shift(r2, kMaxG), -30);
  uint16_t* slot = reinterpret_cast<uint16_t*>(index + L.slots) + int64_t(b) * kSlotCap;
  uint32_t cnt = 0;
  for (int k0 = 0; k0 < n; k0 += 64) {
    const int k = k0 + lane;
    bool take = false;
    if (k < n) {
      double gk[P];
#pragma unroll
      for (int t = 0; t < P; ++t) gk[t] = double(grid[k * P + t]);
      double dn, dx;
      box_d2<P>(gk, lo, kW, dn, dx);
      take = dn <= u + m;
    }
    const uint64_t bal = __ballot(take);
    if (take) {
      const uint32_t at = cnt + uint32_t(__popcll(bal & ((uint64_t(1) << lane) - 1)));
      if (at < uint32_t(kSlotCap)) slot[at] = uint16_t(k);
    }
    cnt += uint32_t(__popcll(bal));
  }
  if (lane == 0)
    reinterpret_cast<uint16_t*>(index + L.counts)[b] = uint16_t(cnt < 65535u ? cnt : 65535u);
}

// One block of 1024 threads: offsets, the lists back to back, the header.
template <int P, int N>
__global__ __launch_bounds__(1024) void index_finish_kernel(const float* __restrict__ grid, int n,
                                                            uint8_t* __restrict__ index) {
  using B = Buckets<P, N>;
  constexpr int kThreads = 1024;
  const IndexLayout L = index_layout(P, n);
  __shared__ uint32_t s_off[B::kCells + 1];
  __shared__ uint32_t s_tmp[kThreads / 64];
  __shared__ uint64_t s_hash[kThreads / 64];
  __shared__ double s_r2[kThreads / 64];
  __shared__ int s_over;
  const int tid = int(threadIdx.x), lane = tid & 63, wave = tid >> 6;
  const uint16_t* counts = reinterpret_cast<const uint16_t*>(index + L.counts);
  const uint16_t* slots = reinterpret_cast<const uint16_t*>(index + L.slots);
  if (tid == 0) s_over = 0;
  __syncthreads();
  for (int b = tid; b < B::kCells; b += kThreads) {
    const uint32_t c = counts[b];
    if (c > uint32_t(kSlotCap)) s_over = 1;
    s_off[b] = c;
  }
  __syncthreads();
  const int total = block_offsets(s_off, B::kCells, tid, kThreads, s_tmp);
  const bool usable = s_over == 0 && total <= index_list_cap(P, n);
  uint16_t* offs = reinterpret_cast<uint16_t*>(index + L.offsets);
  uint16_t* list = reinterpret_cast<uint16_t*>(index + L.list);
  for (int b = tid; b <= B::kCells; b += kThreads) offs[b] = usable ? uint16_t(s_off[b]) : 0;
  if (usable) {
    for (int b = tid; b < B::kCells; b += kThreads) {
      const uint32_t o = s_off[b], c = s_off[b + 1] - o;
      for (uint32_t e = 0; e < c; ++e) list[o + e] = slots[int64_t(b) * kSlotCap + e];
    }
  }
  uint64_t h = 0;
  double r2 = 0.0;
  for (int k = tid; k < n; k += kThreads) {
    float c[P];
    double s = 0.0;
#pragma unroll
    for (int t = 0; t < P; ++t) {
      c[t] = grid[k * P + t];
      s += double(c[t]) * double(c[t]);
    }
    h += point_hash<P>(c, k);
    r2 = fmax(r2, s);
  }
  h = wave_sum(h, lane);
  r2 = wave_max(r2, lane);
  if (lane == 0) {
    s_hash[wave] = h;
    s_r2[wave] = r2;
  }
  __syncthreads();
  if (tid == 0) {
    uint64_t hs = 0;
    double rr = 0.0;
    for (int w = 0; w < kThreads / 64; ++w) {
      hs += s_hash[w];
      rr = fmax(rr, s_r2[w]);
    }
    IndexHeader hd{};
    hd.magic = kIndexMagic;
    hd.p = P;
    hd.n = uint32_t(n);
    hd.nb = B::kNB;
    hd.total = usable ? uint32_t(total) : 0u;
    hd.usable = usable ? 1u : 0u;
    hd.hash = hs;
    hd.margin = ldexp(search_shift(rr, kMaxG), -30);
    hd.half_side = kBR;
    *reinterpret_cast<IndexHeader*>(index) = hd;
  }
}

// grid point in LDS: its coordinates as read (fp32, exact in fp64), one
// 8-byte read per candidate; the search constant is formed in registers
struct __align__(8) GridPt {
  float x[2];
};

// |G_k|^2 / 2 + S in fp64: the squares are exact, then one rounding for
// their sum (p = 2) and one for adding S (half the sum is exact)
template <int P>
__device__ inline double search_const(const GridPt& q, double shift) {
  double h = double(q.x[0]) * double(q.x[0]);
  if constexpr (P == 2) h = fma(double(q.x[1]), double(q.x[1]), h);
  return fma(0.5, h, shift);
}

__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// E: weights per lane (g = 64 E); P: grid dimension; BITS: packed code width;
// kQW: waves per block. The waves of a block share the grid and the index in
// LDS and then take groups independently (no block barrier after the
// prologue).
template <int E, int P, int BITS, int kQW, typename InT>
__global__ __launch_bounds__(64 * kQW) void quantize_kernel(
    const InT* __restrict__ w, int64_t rows, int64_t in, uint64_t seed,
    const float* __restrict__ grid, int n, const uint8_t* __restrict__ index,
    uint8_t* __restrict__ codes, int64_t row_bytes, uint16_t* __restrict__ scales) {
  constexpr int G = 64 * E;
  constexpr int kVecPerLane = E / P;
  constexpr int kCodesPerGroup = G / P;
  constexpr int kWordsPerGroup = kCodesPerGroup * BITS / 32;
  static_assert(E % P == 0, "a lane must hold whole p-vectors");
  static_assert(E <= 16, "groups above 1024 weights take quantize_scan_kernel");
  static_assert((kCodesPerGroup * BITS) % 32 == 0, "group must fill whole dwords");
  constexpr int kN = 1 << BITS;  // grid points of the format (the host passes n = 2^BITS)
  static_assert(kN <= kMaxN, "grid size");
  using BK = Buckets<P, kN>;
  constexpr int kCap = index_list_cap(P, kN);
  constexpr IndexLayout kL = index_layout(P, kN);
  using CodeT = typename std::conditional<(BITS <= 8), uint8_t, uint16_t>::type;

  __shared__ GridPt s_grid[kN];
  __shared__ CodeT s_codes[kQW][kCodesPerGroup];
  __shared__ __align__(16) uint16_t s_off[align16((BK::kCells + 1) * 2) / 2];
  __shared__ __align__(16) uint16_t s_list[kCap];
  __shared__ double s_r2[kQW];
  __shared__ uint64_t s_hash[kQW];

  const int tid = int(threadIdx.x);
  const int lane = tid & 63;
  const int wave = tid >> 6;

  // the grid, its largest squared norm and (with an index) its hash
  double r2 = 0.0;
  uint64_t hsh = 0;
  for (int k = tid; k < n; k += 64 * kQW) {
    float c[P];
    double h = 0.0;
#pragma unroll
    for (int t = 0; t < P; ++t) {
      c[t] = grid[k * P + t];
      h += double(c[t]) * double(c[t]);
    }
    GridPt q;
    q.x[0] = c[0];
    q.x[1] = P == 2 ? c[P - 1] : 0.0f;
    s_grid[k] = q;
    r2 = fmax(r2, h);
    if (index != nullptr) hsh += point_hash<P>(c, k);
  }
  r2 = wave_max(r2, lane);
  hsh = wave_sum(hsh, lane);
  if (lane == 0) {
    s_r2[wave] = r2;
    s_hash[wave] = hsh;
  }
  __syncthreads();
  hsh = 0;
  for (int i = 0; i < kQW; ++i) {
    r2 = fmax(r2, s_r2[i]);
    hsh += s_hash[i];
  }
  const double shift = search_shift(r2, G);

  // the index, when it was built from this grid and fits
  bool pruned = false;
  if (index != nullptr) {
    const IndexHeader* hd = reinterpret_cast<const IndexHeader*>(index);
    pruned = hd->magic == kIndexMagic && hd->p == uint32_t(P) && hd->n == uint32_t(n) &&
             hd->nb == uint32_t(BK::kNB) && hd->usable == 1u && hd->total <= uint32_t(kCap) &&
             hd->hash == hsh && hd->half_side == kBR && hd->margin >= ldexp(shift, -30);
    if (pruned) {
      const int total = int(hd->total);
      const u32x4* so = reinterpret_cast<const u32x4*>(index + kL.offsets);
      u32x4* d_off = reinterpret_cast<u32x4*>(s_off);
      for (int i = tid; i < int(sizeof(s_off) / 16); i += 64 * kQW) d_off[i] = so[i];
      const u32x4* sl = reinterpret_cast<const u32x4*>(index + kL.list);
      u32x4* d_list = reinterpret_cast<u32x4*>(s_list);
      for (int i = tid; i < (total + 7) / 8; i += 64 * kQW) d_list[i] = sl[i];
    }
  }

  uint64_t neg = 0;
#pragma unroll
  for (int i = 0; i < E; ++i) neg |= uint64_t(rht_sign_negative(seed, uint32_t(lane * E + i))) << i;

  const int64_t groups_per_row = in / G;
  const int64_t total = rows * groups_per_row;
  const double inv_sqrt_g = 1.0 / sqrt(double(G));
  const uint32_t index_mask = kIndexMask;
  __syncthreads();

  for (int64_t grp = int64_t(blockIdx.x) * kQW + wave; grp < total;
       grp += int64_t(gridDim.x) * kQW) {
    const int64_t row = grp / groups_per_row;
    const int64_t gi = grp - row * groups_per_row;

    double v[E];
    load_group<E, InT>(w + row * in + gi * G + lane * E, v);

    double ss = 0.0;
#pragma unroll
    for (int i = 0; i < E; ++i) ss += v[i] * v[i];
    ss = wave_sum(ss, lane);
    const double s = sqrt(ss);

    // w / s as w * (1 / s): within an ulp of the quotient
    const double inv_s = s > 0.0 ? 1.0 / s : 0.0;
#pragma unroll
    for (int i = 0; i < E; ++i) {
      const double u = v[i] * inv_s;
      v[i] = ((neg >> i) & 1) ? -u : u;
    }
    fwht_wave<E>(v, lane, G);

    // search value of point k for vector j, folded into best[j]
    double best[kVecPerLane];
#pragma unroll
    for (int j = 0; j < kVecPerLane; ++j) best[j] = INFINITY;
    auto fold = [&](int j, int k, const GridPt& q) {
      double c = fma(-v[j * P], double(q.x[0]), search_const<P>(q, shift));
      if constexpr (P == 2) c = fma(-v[j * P + 1], double(q.x[1]), c);
      best[j] = min_indexed(best[j], c, uint32_t(k), index_mask);
    };
    // vectors that scan every point (one bit per vector of the lane)
    uint64_t full = (uint64_t(1) << kVecPerLane) - 1;
    if (pruned) {
      // the vectors' lists, walked side by side (a list that ends repeats
      // its last entry, which leaves the minimum unchanged)
      int at[kVecPerLane], last[kVecPerLane];
      int steps = 0;
#pragma unroll
      for (int j = 0; j < kVecPerLane; ++j) {
        int b = bucket_axis(v[j * P], BK::kNB);
        if constexpr (P == 2) {
          const int by = bucket_axis(v[j * P + 1], BK::kNB);
          b = (b < 0 || by < 0) ? -1 : by * BK::kNB + b;
        }
        at[j] = 0;
        last[j] = 0;
        if (b >= 0) {
          const int o = s_off[b], e = s_off[b + 1];
          at[j] = o;
          last[j] = e - o - 1;
          steps = max(steps, e - o);
          full &= ~(uint64_t(1) << j);
        }
      }
      for (int i = 0; i < steps; ++i) {
        // all reads of the step first (the folds below are opaque to the
        // scheduler, so reads placed between them would wait one by one)
        int k[kVecPerLane];
        GridPt q[kVecPerLane];
#pragma unroll
        for (int j = 0; j < kVecPerLane; ++j) k[j] = s_list[at[j] + min(i, last[j])];
#pragma unroll
        for (int j = 0; j < kVecPerLane; ++j) q[j] = s_grid[k[j]];
#pragma unroll
        for (int j = 0; j < kVecPerLane; ++j) fold(j, k[j], q[j]);
      }
    }
    if (full != 0) {
#pragma unroll
      for (int j = 0; j < kVecPerLane; ++j)
        if ((full >> j) & 1)
          for (int k = 0; k < n; ++k) fold(j, k, s_grid[k]);
    }

#pragma unroll
    for (int j = 0; j < kVecPerLane; ++j)
      s_codes[wave][lane * kVecPerLane + j] =
          CodeT(__builtin_bit_cast(uint64_t, best[j]) & kIndexMask);
    wave_sync();
    uint32_t* dst = reinterpret_cast<uint32_t*>(codes + row * row_bytes +
                                                gi * (int64_t(kCodesPerGroup) * BITS / 8));
    for (int wi = lane; wi < kWordsPerGroup; wi += 64) {
      const int bit0 = wi * 32;
      int c = bit0 / BITS;
      uint32_t word = uint32_t(s_codes[wave][c]) >> (bit0 - c * BITS);
      for (++c; c * BITS < bit0 + 32 && c < kCodesPerGroup; ++c)
        word |= uint32_t(s_codes[wave][c]) << (c * BITS - bit0);
      dst[wi] = word;
    }
    if (lane == 0) scales[row * groups_per_row + gi] = f64_to_f16_rne(s * inv_sqrt_g);
    wave_sync();
  }
}

// Groups of 2048 and 4096 weights (E = 32, 64): every vector scans all n
// points, the waves of a block step through groups together. The candidate
// walk of quantize_kernel is not used at these sizes: its build for p = 2,
// g = 4096 (32 vectors per lane, registers spilled to the accumulation
// registers) did not finish on the GPU, and the cause has not been found.
template <int E, int P, int BITS, typename InT>
__global__ __launch_bounds__(64 * kWaves) void quantize_scan_kernel(
    const InT* __restrict__ w, int64_t rows, int64_t in, uint64_t seed,
    const float* __restrict__ grid, int n, uint8_t* __restrict__ codes, int64_t row_bytes,
    uint16_t* __restrict__ scales) {
  constexpr int G = 64 * E;
  constexpr int kVecPerLane = E / P;
  constexpr int kCodesPerGroup = G / P;
  constexpr int kWordsPerGroup = kCodesPerGroup * BITS / 32;
  static_assert(E % P == 0, "a lane must hold whole p-vectors");
  static_assert((kCodesPerGroup * BITS) % 32 == 0, "group must fill whole dwords");

  // grid point k: P coordinates then |G_k|^2 / 2 + shift (stride P + 1)
  __shared__ double s_grid[kMaxN * (P + 1)];
  __shared__ uint16_t s_codes[kWaves][kMaxG / P];

  const int lane = int(threadIdx.x) & 63;
  const int wave = int(threadIdx.x) >> 6;

  __shared__ double s_r2[kWaves];
  double r2 = 0.0;  // largest squared grid-point norm seen by this thread
  for (int k = int(threadIdx.x); k < n; k += 64 * kWaves) {
    double h = 0.0;
#pragma unroll
    for (int t = 0; t < P; ++t) {
      const double c = double(grid[k * P + t]);
      s_grid[k * (P + 1) + t] = c;
      h += c * c;
    }
    s_grid[k * (P + 1) + P] = 0.5 * h;
    r2 = fmax(r2, h);
  }
  r2 = wave_max(r2, int(threadIdx.x) & 63);
  if ((threadIdx.x & 63) == 0) s_r2[threadIdx.x >> 6] = r2;
  __syncthreads();
  for (int w = 0; w < kWaves; ++w) r2 = fmax(r2, s_r2[w]);
  // the search-value shift: a power of two at least twice the largest |c_k|
  const double bound = 2.0 * (0.5 * r2 + sqrt(double(64 * E)) * sqrt(r2));
  const double shift = bound <= kMinShift ? kMinShift : exp2(ceil(log2(bound)));
  for (int k = int(threadIdx.x); k < n; k += 64 * kWaves) s_grid[k * (P + 1) + P] += shift;

  uint64_t neg = 0;
#pragma unroll
  for (int i = 0; i < E; ++i) neg |= uint64_t(rht_sign_negative(seed, uint32_t(lane * E + i))) << i;

  const int64_t groups_per_row = in / G;
  const int64_t total = rows * groups_per_row;
  const double inv_sqrt_g = 1.0 / sqrt(double(G));
  __syncthreads();

  // Every wave of the block runs the same number of iterations (barriers).
  for (int64_t first = int64_t(blockIdx.x) * kWaves; first < total;
       first += int64_t(gridDim.x) * kWaves) {
    const int64_t grp = first + wave;
    const bool valid = grp < total;
    const int64_t row = valid ? grp / groups_per_row : 0;
    const int64_t gi = valid ? grp - row * groups_per_row : 0;

    double v[E];
    if (valid) {
      load_group<E, InT>(w + row * in + gi * G + lane * E, v);
    } else {
#pragma unroll
      for (int i = 0; i < E; ++i) v[i] = 0.0;
    }

    double ss = 0.0;
#pragma unroll
    for (int i = 0; i < E; ++i) ss += v[i] * v[i];
    ss = wave_sum(ss, lane);
    const double s = sqrt(ss);

#pragma unroll
    for (int i = 0; i < E; ++i) {
      const double u = s > 0.0 ? v[i] / s : 0.0;
      v[i] = ((neg >> i) & 1) ? -u : u;
    }
    fwht_wave<E>(v, lane, G);

    double best[kVecPerLane];
#pragma unroll
    for (int j = 0; j < kVecPerLane; ++j) best[j] = INFINITY;
    const uint32_t index_mask = kIndexMask;
    for (int k = 0; k < n; ++k) {
      double gk[P];
#pragma unroll
      for (int t = 0; t < P; ++t) gk[t] = s_grid[k * (P + 1) + t];
      const double hk = s_grid[k * (P + 1) + P];
#pragma unroll
      for (int j = 0; j < kVecPerLane; ++j) {
        double c = hk;
#pragma unroll
        for (int t = 0; t < P; ++t) c = fma(-v[j * P + t], gk[t], c);
        best[j] = min_indexed(best[j], c, uint32_t(k), index_mask);
      }
    }

#pragma unroll
    for (int j = 0; j < kVecPerLane; ++j)
      s_codes[wave][lane * kVecPerLane + j] =
          uint16_t(__builtin_bit_cast(uint64_t, best[j]) & kIndexMask);
    __syncthreads();

    if (valid) {
      uint32_t* dst = reinterpret_cast<uint32_t*>(codes + row * row_bytes +
                                                  gi * (int64_t(kCodesPerGroup) * BITS / 8));
      for (int wi = lane; wi < kWordsPerGroup; wi += 64) {
        const int bit0 = wi * 32;
        int c = bit0 / BITS;
        uint32_t word = uint32_t(s_codes[wave][c]) >> (bit0 - c * BITS);
        for (++c; c * BITS < bit0 + 32 && c < kCodesPerGroup; ++c)
          word |= uint32_t(s_codes[wave][c]) << (c * BITS - bit0);
        dst[wi] = word;
      }
      if (lane == 0) scales[row * groups_per_row + gi] = f64_to_f16_rne(s * inv_sqrt_g);
    }
    __syncthreads();
  }
}


// Quantization error of a layer, measured in the rotated space: the rotation
// R = H diag(sigma) / sqrt(g) is orthonormal, so per group (Parseval)
//   ||w - w_hat||^2 = || H (sigma * w) / sqrt(g) - scale * concat_j G[code_j] ||^2
// with w_hat the dequantised group (App. G). One wavefront per group writes
// that sum and ||w||^2 as two fp64 values (row-major group order); the layer's
// relative error t^2 (Sec. 3.4) is their ratio of sums. Codes are read from
// the packed row (LSB-first, `bits` per code, up to three bytes per code).
template <int E, int P, typename InT>
__global__ __launch_bounds__(64 * kWaves) void layer_error_kernel(
    const InT* __restrict__ w, int64_t rows, int64_t in, uint64_t seed,
    const float* __restrict__ grid, int bits, const uint8_t* __restrict__ codes, int64_t row_bytes,
    const uint16_t* __restrict__ scales, double* __restrict__ out) {
  constexpr int G = 64 * E;
  static_assert(E % P == 0, "a lane must hold whole p-vectors");
  const int lane = int(threadIdx.x) & 63;
  const int wave = int(threadIdx.x) >> 6;
  uint64_t neg = 0;
#pragma unroll
  for (int i = 0; i < E; ++i) neg |= uint64_t(rht_sign_negative(seed, uint32_t(lane * E + i))) << i;
  const int64_t groups_per_row = in / G;
  const int64_t total = rows * groups_per_row;
  const double inv_sqrt_g = 1.0 / sqrt(double(G));
  const uint32_t mask = (1u << bits) - 1u;
  // no barrier below: each wave walks its own groups
  for (int64_t grp = int64_t(blockIdx.x) * kWaves + wave; grp < total;
       grp += int64_t(gridDim.x) * kWaves) {
    const int64_t row = grp / groups_per_row;
    const int64_t gi = grp - row * groups_per_row;
    double v[E];
    load_group<E, InT>(w + row * in + gi * G + lane * E, v);
    double ss = 0.0;
#pragma unroll
    for (int i = 0; i < E; ++i) ss += v[i] * v[i];
    ss = wave_sum(ss, lane);
#pragma unroll
    for (int i = 0; i < E; ++i)
      if ((neg >> i) & 1) v[i] = -v[i];
    fwht_wave<E>(v, lane, G);
    const double sh = double(__builtin_bit_cast(_Float16, scales[row * groups_per_row + gi]));
    const uint8_t* crow = codes + row * row_bytes;
    double e = 0.0;
#pragma unroll
    for (int t = 0; t < E / P; ++t) {
      const int64_t m = gi * (G / P) + lane * (E / P) + t;  // code index in the row
      const int64_t bit = m * bits;
      const int64_t b0 = bit >> 3;
      uint32_t win = crow[b0];
      if (b0 + 1 < row_bytes) win |= uint32_t(crow[b0 + 1]) << 8;
      if (b0 + 2 < row_bytes) win |= uint32_t(crow[b0 + 2]) << 16;
      const uint32_t code = (win >> (bit & 7)) & mask;
#pragma unroll
      for (int c = 0; c < P; ++c) {
        const double d = v[t * P + c] * inv_sqrt_g - sh * double(grid[code * P + c]);
        e += d * d;
      }
    }
    e = wave_sum(e, lane);
    if (lane == 0) {
      out[2 * grp] = e;
      out[2 * grp + 1] = ss;
    }
  }
}

// t^2 = sum_q err_q / sum_q norm_q over the per-group pairs of
// layer_error_kernel (Sec. 3.4's relative error of the layer). One block:
// thread t adds the pairs t, t + 256, ... in order, then a fixed tree over
// the threads (deterministic). A layer of norm 0 gets t^2 = 0.
__global__ __launch_bounds__(256) void layer_t2_kernel(const double* __restrict__ pairs,
                                                       int64_t groups, double* __restrict__ t2) {
  __shared__ double s_e[256], s_n[256];
  const int tid = int(threadIdx.x);
  double e = 0.0, nrm = 0.0;
  for (int64_t q = tid; q < groups; q += 256) {
    e += pairs[2 * q];
    nrm += pairs[2 * q + 1];
  }
  s_e[tid] = e;
  s_n[tid] = nrm;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (tid < h) {
      s_e[tid] += s_e[tid + h];
      s_n[tid] += s_n[tid + h];
    }
    __syncthreads();
  }
  if (tid == 0) t2[0] = s_n[0] > 0.0 ? s_e[0] / s_n[0] : 0.0;
}

template <int P, typename InT>
hipError_t launch_error_p(const InT* w, int64_t out_rows, int64_t in, const float* grid, int bits,
                          int g, uint64_t seed, const uint8_t* codes, int64_t row_bytes,
                          const uint16_t* scales, double* err, hipStream_t stream) {
  const int64_t total = out_rows * (in / g);
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((total + kWaves - 1) / kWaves, 8192));
  const dim3 grid_dim{unsigned(blocks)}, block{64 * kWaves};
  switch (g) {
#define HIGGS_E_CASE(GV)                                                                     \
  case GV:                                                                                   \
    if constexpr ((GV / 64) % P == 0) {                                                      \
      hipLaunchKernelGGL((layer_error_kernel<GV / 64, P, InT>), grid_dim, block, 0, stream, \
                         w, out_rows, in, seed, grid, bits, codes, row_bytes, scales, err);  \
      return hipGetLastError();                                                              \
    }                                                                                        \
    break;
    HIGGS_E_CASE(64)
    HIGGS_E_CASE(128)
    HIGGS_E_CASE(256)
    HIGGS_E_CASE(512)
    HIGGS_E_CASE(1024)
    HIGGS_E_CASE(2048)
    HIGGS_E_CASE(4096)
#undef HIGGS_E_CASE
    default:
      break;
  }
  return hipErrorInvalidValue;
}

template <int P, int BITS, typename InT>
hipError_t launch_bits(const InT* w, int64_t out, int64_t in, const float* grid, int n,
                       const uint8_t* index, int g, uint64_t seed, uint8_t* codes,
                       int64_t row_bytes, uint16_t* scales, hipStream_t stream) {
  const int64_t total = out * (in / g);
  // a block loads the grid and the index into LDS once, then its waves
  // take groups in turn. The 1024-point grid's index fills a compute unit's
  // LDS, and scalar grids run 2 waves per SIMD (registers): there one block
  // per compute unit with 12 or 8 waves; else blocks of 4 waves, up to 2048
  // (measured faster there)
  constexpr int kQW = P == 1 ? 8 : (BITS >= 8 ? 12 : 4);
  constexpr int64_t kMaxBlocks = kQW == 4 ? 2048 : 256;
  const int64_t blocks =
      std::max<int64_t>(1, std::min<int64_t>((total + kQW - 1) / kQW, kMaxBlocks));
  const dim3 grid_dim{unsigned(blocks)}, block{64 * kQW}, scan_block{64 * kWaves};
  switch (g) {
#define HIGGS_Q_CASE(GV)                                                                     \
  case GV:                                                                                   \
    if constexpr ((GV / 64) % P == 0) {                                                      \
      hipLaunchKernelGGL((quantize_kernel<GV / 64, P, BITS, kQW, InT>), grid_dim, block, 0,  \
                         stream, w, out, in, seed, grid, n, index, codes, row_bytes,         \
                         scales);                                                            \
      return hipGetLastError();                                                              \
    }                                                                                        \
    break;
    HIGGS_Q_CASE(64)
    HIGGS_Q_CASE(128)
    HIGGS_Q_CASE(256)
    HIGGS_Q_CASE(512)
    HIGGS_Q_CASE(1024)
#undef HIGGS_Q_CASE
    default:
      break;
  }
  // larger groups: the full scan, one block per four groups
  const dim3 scan_grid{unsigned(std::min<int64_t>((total + kWaves - 1) / kWaves, 8192))};
  switch (g) {
#define HIGGS_S_CASE(GV)                                                                     \
  case GV:                                                                                   \
    if constexpr ((GV / 64) % P == 0) {                                                      \
      hipLaunchKernelGGL((quantize_scan_kernel<GV / 64, P, BITS, InT>), scan_grid,           \
                         scan_block, 0, stream, w, out, in, seed, grid, n, codes, row_bytes, \
                         scales);                                                            \
      return hipGetLastError();                                                              \
    }                                                                                        \
    break;
    HIGGS_S_CASE(2048)
    HIGGS_S_CASE(4096)
#undef HIGGS_S_CASE
    default:
      break;
  }
  return hipErrorInvalidValue;
}

template <typename InT>
hipError_t launch_typed(const InT* w, int64_t out, int64_t in, const float* grid, int p, int n,
                        const uint8_t* index, int g, uint64_t seed, uint8_t* codes,
                        uint16_t* scales, hipStream_t stream) {
  const int bits = code_bits(p, n);
  const int64_t row_bytes = in / p * bits / 8;
  if (p == 1 && bits == 4)
    return launch_bits<1, 4>(w, out, in, grid, n, index, g, seed, codes, row_bytes,
                             scales, stream);
  if (p == 1 && bits == 8)
    return launch_bits<1, 8>(w, out, in, grid, n, index, g, seed, codes, row_bytes,
                             scales, stream);
  if (p == 2 && bits == 6)
    return launch_bits<2, 6>(w, out, in, grid, n, index, g, seed, codes, row_bytes,
                             scales, stream);
  if (p == 2 && bits == 8)
    return launch_bits<2, 8>(w, out, in, grid, n, index, g, seed, codes, row_bytes,
                             scales, stream);
  if (p == 2 && bits == 10)
    return launch_bits<2, 10>(w, out, in, grid, n, index, g, seed, codes, row_bytes,
                              scales, stream);
  return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// GPTQ rounding in place of the nearest-point step (Sec. 3.5), in the rotated
// space: W' = per group H (sigma * w) / sqrt(g), the Hessian of the rotated
// calibration activations, U the upper Cholesky factor of its damped inverse
// (Hinv = U^T U). Columns are taken in order, one p-vector at a time: its
// rotated weights v are rounded like Alg. 1 (nearest grid point of
// v sqrt(g) / s, s the group's norm), the error e = v - (s / sqrt(g)) G[q] is
// scaled, E = e U_pp^-1 (U_pp the p x p diagonal block), and later columns
// move by -E U[p-vector, later]. Within a block of 64 columns the update runs
// here, one wavefront per row (lane j holds column c0 + j); the block's E go
// to `err` and the columns after the block are updated by one GEMM.
// ---------------------------------------------------------------------------

// Rotated weights W' (fp64), each group's norm s (fp64) and the stored scale
// fp16(s / sqrt(g)). One wavefront per group.
template <int E, typename InT>
__global__ __launch_bounds__(64 * kWaves) void gptq_prepare_kernel(
    const InT* __restrict__ w, int64_t rows, int64_t in, uint64_t seed, double* __restrict__ wr,
    double* __restrict__ norms, uint16_t* __restrict__ scales) {
  constexpr int G = 64 * E;
  const int lane = int(threadIdx.x) & 63;
  const int wave = int(threadIdx.x) >> 6;
  uint64_t neg = 0;
#pragma unroll
  for (int i = 0; i < E; ++i) neg |= uint64_t(rht_sign_negative(seed, uint32_t(lane * E + i))) << i;
  const int64_t groups_per_row = in / G;
  const int64_t total = rows * groups_per_row;
  const double inv_sqrt_g = 1.0 / sqrt(double(G));
  for (int64_t grp = int64_t(blockIdx.x) * kWaves + wave; grp < total;
       grp += int64_t(gridDim.x) * kWaves) {
    const int64_t row = grp / groups_per_row;
    const int64_t gi = grp - row * groups_per_row;
    double v[E];
    load_group<E, InT>(w + row * in + gi * G + lane * E, v);
    double ss = 0.0;
#pragma unroll
    for (int i = 0; i < E; ++i) ss += v[i] * v[i];
    ss = wave_sum(ss, lane);
    const double sn = sqrt(ss);
#pragma unroll
    for (int i = 0; i < E; ++i)
      if ((neg >> i) & 1) v[i] = -v[i];
    fwht_wave<E>(v, lane, G);
    double* dst = wr + row * in + gi * G + lane * E;
#pragma unroll
    for (int i = 0; i < E; ++i) dst[i] = v[i] * inv_sqrt_g;
    if (lane == 0) {
      norms[grp] = sn;
      scales[grp] = f64_to_f16_rne(sn * inv_sqrt_g);
    }
  }
}

__device__ inline double readlane_f64(double v, int l) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(u)), l));
  const uint32_t hi = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(u >> 32)), l));
  return __builtin_bit_cast(double, uint64_t(lo) | (uint64_t(hi) << 32));
}

// One block of 64 columns [c0, c0 + 64) for every row (one wavefront per row).
template <int P>
__global__ __launch_bounds__(64 * kWaves) void gptq_block_kernel(
    const double* __restrict__ wr, const double* __restrict__ norms,
    const double* __restrict__ u, const float* __restrict__ grid, int n, int64_t rows,
    int64_t in, int log2g, int64_t c0, int bits, uint8_t* __restrict__ codes, int64_t row_bytes,
    double* __restrict__ err) {
  constexpr int kB = 64;
  constexpr int kVecs = kB / P;
  __shared__ double s_u[kB][kB + 1];
  __shared__ double s_grid[kMaxN * (P + 1)];
  __shared__ uint16_t s_codes[kWaves][kVecs];
  const int tid = int(threadIdx.x);
  const int lane = tid & 63;
  const int wave = tid >> 6;
  for (int i = tid; i < kB * kB; i += 64 * kWaves) {
    const int r = i / kB, c = i % kB;
    s_u[r][c] = c >= r ? u[(c0 + r) * in + c0 + c] : 0.0;  // upper triangle only
  }
  for (int k = tid; k < n; k += 64 * kWaves) {
    double h = 0.0;
#pragma unroll
    for (int t = 0; t < P; ++t) {
      const double c = double(grid[k * P + t]);
      s_grid[k * (P + 1) + t] = c;
      h += c * c;
    }
    s_grid[k * (P + 1) + P] = 0.5 * h;
  }
  __syncthreads();
  const int64_t row = int64_t(blockIdx.x) * kWaves + wave;
  if (row >= rows) return;  // no barrier below
  const int g = 1 << log2g;
  const double sn = norms[row * (in >> log2g) + (c0 >> log2g)];  // the block is in one group
  const double fwd = sn > 0.0 ? sqrt(double(g)) / sn : 0.0;      // W' -> grid units
  const double back = sn / sqrt(double(g));                      // grid units -> W'
  double wv = wr[row * in + c0 + lane];
  double my_err = 0.0;
  for (int t = 0; t < kVecs; ++t) {
    double v[P], uv[P];
#pragma unroll
    for (int k = 0; k < P; ++k) {
      v[k] = readlane_f64(wv, t * P + k);
      uv[k] = v[k] * fwd;
    }
    // nearest grid point: lane l scans candidates l, l + 64, ...; then the
    // wave keeps the least (c, index) pair (lowest index on ties)
    double best = INFINITY;
    int bk = 0;
    for (int k = lane; k < n; k += 64) {
      double c = s_grid[k * (P + 1) + P];
#pragma unroll
      for (int d = 0; d < P; ++d) c = fma(-uv[d], s_grid[k * (P + 1) + d], c);
      if (c < best) {
        best = c;
        bk = k;
      }
    }
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) {
      const double ob = __shfl_xor(best, m, 64);
      const int ok = __shfl_xor(bk, m, 64);
      if (ob < best || (ob == best && ok < bk)) {
        best = ob;
        bk = ok;
      }
    }
    const int q = __builtin_amdgcn_readfirstlane(bk);
    double e[P], es[P];
#pragma unroll
    for (int k = 0; k < P; ++k) e[k] = v[k] - back * s_grid[q * (P + 1) + k];
    // E = e U_pp^-1 (U_pp upper triangular)
    const int i0 = t * P;
    if constexpr (P == 1) {
      es[0] = e[0] / s_u[i0][i0];
    } else {
      es[0] = e[0] / s_u[i0][i0];
      es[1] = (e[1] - es[0] * s_u[i0][i0 + 1]) / s_u[i0 + 1][i0 + 1];
    }
    if (lane >= i0 + P) {
#pragma unroll
      for (int k = 0; k < P; ++k) wv = fma(-es[k], s_u[i0 + k][lane], wv);
    }
#pragma unroll
    for (int k = 0; k < P; ++k)
      if (lane == i0 + k) my_err = es[k];
    if (lane == 0) s_codes[wave][t] = uint16_t(q);
  }
  err[row * kB + lane] = my_err;
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  // pack the block's codes: kVecs * bits bits, whole dwords
  const int words = kVecs * bits / 32;
  uint32_t* dst = reinterpret_cast<uint32_t*>(codes + row * row_bytes + (c0 / P) * bits / 8);
  if (lane < words) {
    const int bit0 = lane * 32;
    int c = bit0 / bits;
    uint32_t word = uint32_t(s_codes[wave][c]) >> (bit0 - c * bits);
    for (++c; c * bits < bit0 + 32 && c < kVecs; ++c)
      word |= uint32_t(s_codes[wave][c]) << (c * bits - bit0);
    dst[lane] = word;
  }
}

__global__ void f32_to_f64_kernel(const float* __restrict__ src, int64_t count,
                                  double* __restrict__ dst) {
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < count;
       i += int64_t(gridDim.x) * 256)
    dst[i] = double(src[i]);
}

// h[i][i] += damp * mean_i h[i][i] (one block; the mean is summed in a fixed
// order: each thread a strided partial, then thread 0 over the partials)
__global__ __launch_bounds__(256) void damp_diag_kernel(double* __restrict__ h, int64_t in,
                                                        double damp) {
  __shared__ double s_part[256];
  double sum = 0.0;
  for (int64_t i = threadIdx.x; i < in; i += 256) sum += h[i * in + i];
  s_part[threadIdx.x] = sum;
  __syncthreads();
  __shared__ double s_add;
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int k = 0; k < 256; ++k) t += s_part[k];
    s_add = damp * t / double(in);
  }
  __syncthreads();
  for (int64_t i = threadIdx.x; i < in; i += 256) h[i * in + i] += s_add;
}

}  // namespace

hipError_t launch_gptq_prepare(const void* w, higgs_dtype dtype, int64_t out, int64_t in, int g,
                               uint64_t seed, double* wr, double* norms, uint16_t* scales,
                               hipStream_t stream) {
  const int64_t total = out * (in / g);
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((total + kWaves - 1) / kWaves, 8192));
  switch (g) {
#define HIGGS_G_CASE(GV)                                                                        \
  case GV:                                                                                      \
    if (dtype == HIGGS_F32)                                                                     \
      hipLaunchKernelGGL((gptq_prepare_kernel<GV / 64, float>), dim3(unsigned(blocks)),        \
                         dim3(64 * kWaves), 0, stream, static_cast<const float*>(w), out, in,  \
                         seed, wr, norms, scales);                                              \
    else                                                                                        \
      hipLaunchKernelGGL((gptq_prepare_kernel<GV / 64, uint16_t>), dim3(unsigned(blocks)),     \
                         dim3(64 * kWaves), 0, stream, static_cast<const uint16_t*>(w), out,   \
                         in, seed, wr, norms, scales);                                          \
    return hipGetLastError();
    HIGGS_G_CASE(64)
    HIGGS_G_CASE(128)
    HIGGS_G_CASE(256)
    HIGGS_G_CASE(512)
    HIGGS_G_CASE(1024)
    HIGGS_G_CASE(2048)
    HIGGS_G_CASE(4096)
#undef HIGGS_G_CASE
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_gptq_block(const double* wr, const double* norms, const double* u,
                             const float* grid, int p, int n, int64_t out, int64_t in, int g,
                             int64_t c0, uint8_t* codes, double* err, hipStream_t stream) {
  const int bits = code_bits(p, n);
  const int64_t row_bytes = in / p * bits / 8;
  const dim3 grid_dim{unsigned((out + kWaves - 1) / kWaves)}, block{64 * kWaves};
  if (p == 1)
    hipLaunchKernelGGL((gptq_block_kernel<1>), grid_dim, block, 0, stream, wr, norms, u, grid, n,
                       out, in, log2_exact(g), c0, bits, codes, row_bytes, err);
  else
    hipLaunchKernelGGL((gptq_block_kernel<2>), grid_dim, block, 0, stream, wr, norms, u, grid, n,
                       out, in, log2_exact(g), c0, bits, codes, row_bytes, err);
  return hipGetLastError();
}

hipError_t launch_to_f64(const float* src, int64_t count, double* dst, hipStream_t stream) {
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((count + 255) / 256, 8192));
  hipLaunchKernelGGL(f32_to_f64_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream, src, count,
                     dst);
  return hipGetLastError();
}

hipError_t launch_damp_diag(double* h, int64_t in, double damp, hipStream_t stream) {
  hipLaunchKernelGGL(damp_diag_kernel, dim3(1), dim3(256), 0, stream, h, in, damp);
  return hipGetLastError();
}

hipError_t launch_layer_error(const void* w, higgs_dtype dtype, int64_t out, int64_t in,
                              const uint8_t* codes, const uint16_t* scales, const float* grid,
                              int p, int n, int g, uint64_t seed, double* err, double* t2,
                              hipStream_t stream) {
  const int bits = code_bits(p, n);
  const int64_t row_bytes = in / p * bits / 8;
  hipError_t st;
  if (dtype == HIGGS_F32) {
    const float* wf = static_cast<const float*>(w);
    st = p == 1 ? launch_error_p<1>(wf, out, in, grid, bits, g, seed, codes, row_bytes, scales,
                                    err, stream)
                : launch_error_p<2>(wf, out, in, grid, bits, g, seed, codes, row_bytes, scales,
                                    err, stream);
  } else {
    const uint16_t* wb = static_cast<const uint16_t*>(w);
    st = p == 1 ? launch_error_p<1>(wb, out, in, grid, bits, g, seed, codes, row_bytes, scales,
                                    err, stream)
                : launch_error_p<2>(wb, out, in, grid, bits, g, seed, codes, row_bytes, scales,
                                    err, stream);
  }
  if (st != hipSuccess || t2 == nullptr) return st;
  hipLaunchKernelGGL(layer_t2_kernel, dim3(1), dim3(256), 0, stream, err, out * (in / g), t2);
  return hipGetLastError();
}

hipError_t launch_quantize(const void* w, higgs_dtype dtype, int64_t out, int64_t in,
                           const float* grid, int p, int n, const void* index, int g,
                           uint64_t seed, uint8_t* codes, uint16_t* scales, hipStream_t stream) {
  const uint8_t* idx = static_cast<const uint8_t*>(index);
  if (dtype == HIGGS_F32)
    return launch_typed(static_cast<const float*>(w), out, in, grid, p, n, idx, g, seed, codes,
                        scales, stream);
  return launch_typed(static_cast<const uint16_t*>(w), out, in, grid, p, n, idx, g, seed, codes,
                      scales, stream);
}

int64_t search_index_bytes(int p, int n) { return index_layout(p, n).bytes; }

hipError_t launch_search_index(const float* grid, int p, int n, void* index, hipStream_t stream) {
  uint8_t* idx = static_cast<uint8_t*>(index);
  const dim3 slots_grid{unsigned((index_cells(p, n) + 3) / 4)}, slots_block{256};
#define HIGGS_I_CASE(PV, NV)                                                                 \
  if (p == PV && n == NV) {                                                                  \
    hipLaunchKernelGGL((index_slots_kernel<PV, NV>), slots_grid, slots_block, 0, stream, grid, \
                       n, idx);                                                              \
    hipLaunchKernelGGL((index_finish_kernel<PV, NV>), dim3(1), dim3(1024), 0, stream, grid, n, \
                       idx);                                                                 \
    return hipGetLastError();                                                                \
  }
  HIGGS_I_CASE(1, 16)
  HIGGS_I_CASE(1, 256)
  HIGGS_I_CASE(2, 64)
  HIGGS_I_CASE(2, 256)
  HIGGS_I_CASE(2, 1024)
#undef HIGGS_I_CASE
  return hipErrorInvalidValue;
}

}  // namespace higgs
