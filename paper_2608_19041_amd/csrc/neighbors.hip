// Cell-list neighbour search and the reverse index of a skin list, Methods
// Eq. (neighbor-set), integer arithmetic only.
//
// Positions are mapped to fixed point Q(x) = rint(x * 2^20) (int64) and the
// membership test |Q(r_j) + sum_b n_b Q(h_b) - Q(r_i)|^2 < Q(r)^2 is exact, so
// every list built here is a deterministic function of the float64 positions.
// Rows come out in canonical order (ascending j, then n_x, n_y, n_z).
//
// Binning: positions are wrapped into the cell by integer multiples of the
// quantised lattice vectors, which keeps the test exact.  A diagonal cell is
// binned in integers; a triclinic cell by fractional coordinates in float64,
// which only decides the candidate set: its stencil reach carries a 1e-6 A
// margin, far above the rounding of the fractional coordinates, so every
// pair within the radius is visited and the integer test decides.
//
// Bins are about half the radius wide (reach 2), so a centre's stencil
// covers ~15.6 r^3 instead of 27 r^3 with radius-wide bins.  After binning,
// each atom's fixed-point position and index are copied into a record in bin
// order, so the atoms of consecutive bins along the third axis are one
// contiguous run: the stencil of a centre is a few dozen such runs, which a
// wave reads with coalesced loads as one list of candidates, 64 at a time.
//
// Work mapping: one 64-lane wavefront per centre atom, waves striding over
// centres.  The count kernel counts a row; the fill kernel collects the
// accepted keys (j, packed n) of a row in LDS and writes each at its rank,
// the number of smaller keys in the row: canonical order without a sort
// network.  Rows longer than kMaxRow are ranked the same way from a global
// scratch the host provides once the count has shown them.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "../../include/dpa4c.h"
#include "launch.h"

namespace dpa4c {

namespace {

constexpr int kBlock = 256;            // 4 waves
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kMaxRow = 512;           // longest row the fill kernel ranks in LDS
constexpr int kRankBlock = 8;          // keys compared per step of the bucketed rank
constexpr int kMaxSeg = kWave;         // stencil runs a wave holds at once
constexpr int64_t kFlagCapacity = 1, kFlagRowTooLong = 2, kFlagShift = 4, kFlagNonFinite = 8;
constexpr int kFlagMaxRow = 3;         // flags[3]: the longest row of the last count

__device__ inline int64_t floor_div(int64_t a, int64_t b) {
  int64_t q = a / b;
  return (a % b != 0 && ((a < 0) != (b < 0))) ? q - 1 : q;
}

__device__ inline int64_t qfix(double x) { return static_cast<int64_t>(__builtin_rint(x * kQScale)); }

__device__ inline int lane_id() { return threadIdx.x & (kWave - 1); }

// exclusive prefix count of ``pred`` over the lanes below this one
__device__ inline int ballot_prefix(bool pred, uint64_t* mask_out) {
  uint64_t m = __ballot(pred);
  *mask_out = m;
  return __popcll(m & ((uint64_t(1) << lane_id()) - 1));
}

__device__ inline void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// The same for LDS alone: outstanding global loads and stores of the wave
// are not waited for.
__device__ inline void wave_local_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

struct GridDev {
  int64_t qh[9];          // Q(h_b) in row b
  double inv[9];          // inverse lattice matrix (triclinic binning)
  int nc0, nc1, nc2;
  int re0, re1, re2;
  int64_t rq;
};

GridDev to_dev(const CellGrid& g) {
  GridDev d;
  for (int k = 0; k < 9; ++k) {
    d.qh[k] = g.qh[k];
    d.inv[k] = g.inv[k];
  }
  d.nc0 = g.nc[0];
  d.nc1 = g.nc[1];
  d.nc2 = g.nc[2];
  d.re0 = g.reach[0];
  d.re1 = g.reach[1];
  d.re2 = g.reach[2];
  d.rq = g.rq;
  return d;
}

// within (strictly) the fixed-point radius; no overflow: components are
// rejected before squaring
__device__ inline bool within(int64_t dx, int64_t dy, int64_t dz, int64_t rq) {
  if (dx >= rq || dx <= -rq || dy >= rq || dy <= -rq || dz >= rq || dz <= -rq) return false;
  return dx * dx + dy * dy + dz * dz < rq * rq;
}

// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(kBlock) zero_i32_kernel(int32_t* __restrict__ p, int64_t n) {
  int64_t i = blockIdx.x * int64_t(kBlock) + threadIdx.x;
  if (i < n) p[i] = 0;
}

// qpos = the position wrapped into the cell, Q(x) - sum_b m_b Q(h_b);
// wrap = m; cell_of = its bin
template <bool TRIC>
__global__ void __launch_bounds__(kBlock) bin_kernel(const double* __restrict__ pos, int64_t n,
                                                     GridDev g, int64_t* __restrict__ qpos,
                                                     int32_t* __restrict__ wrap,
                                                     int32_t* __restrict__ cell_of,
                                                     int32_t* __restrict__ cell_cnt,
                                                     int64_t* __restrict__ flags) {
  int64_t i = blockIdx.x * int64_t(kBlock) + threadIdx.x;
  if (i >= n) return;
  const int nc[3] = {g.nc0, g.nc1, g.nc2};
  int c[3];
  bool bad = false;
  double x[3];
  for (int a = 0; a < 3; ++a) {
    x[a] = pos[3 * i + a];
    if (!isfinite(x[a]) || fabs(x[a]) > 1.0e12) {
      bad = true;
      x[a] = 0.0;
    }
  }
  if (!TRIC) {
    for (int a = 0; a < 3; ++a) {
      const int64_t L = g.qh[4 * a];
      int64_t q = qfix(x[a]);
      int64_t m = floor_div(q, L);
      int64_t qw = q - m * L;
      qpos[3 * i + a] = qw;
      wrap[3 * i + a] = static_cast<int32_t>(m);
      c[a] = static_cast<int>((qw * nc[a]) / L);
    }
  } else {
    int64_t m[3];
    double fw[3];
    for (int b = 0; b < 3; ++b) {
      const double f = x[0] * g.inv[b] + x[1] * g.inv[3 + b] + x[2] * g.inv[6 + b];
      const double fl = floor(f);
      m[b] = static_cast<int64_t>(fl);
      fw[b] = f - fl;
    }
    for (int a = 0; a < 3; ++a) {
      qpos[3 * i + a] = qfix(x[a]) - m[0] * g.qh[a] - m[1] * g.qh[3 + a] - m[2] * g.qh[6 + a];
      wrap[3 * i + a] = static_cast<int32_t>(m[a]);
      int cb = static_cast<int>(fw[a] * nc[a]);
      c[a] = cb < 0 ? 0 : (cb >= nc[a] ? nc[a] - 1 : cb);
    }
  }
  if (bad) atomicOr(reinterpret_cast<unsigned long long*>(flags), (unsigned long long)kFlagNonFinite);
  int cid = (c[0] * nc[1] + c[1]) * nc[2] + c[2];
  cell_of[i] = cid;
  atomicAdd(&cell_cnt[cid], 1);
}

// One candidate record per atom, in bin order: the wrapped fixed-point
// position and the atom index (32 bytes, read by two 16-byte loads).
struct alignas(16) CellRec {
  int64_t q[3];
  int32_t j;
  int32_t pad;
};

// the atom's record at a free slot of its bin (slot order inside a bin does
// not matter: rows are ranked by key afterwards)
__global__ void __launch_bounds__(kBlock) place_kernel(int64_t n, const int32_t* __restrict__ cell_of,
                                                       const int64_t* __restrict__ qpos,
                                                       const int32_t* __restrict__ start,
                                                       int32_t* __restrict__ fill,
                                                       CellRec* __restrict__ rec) {
  int64_t i = blockIdx.x * int64_t(kBlock) + threadIdx.x;
  if (i >= n) return;
  int cid = cell_of[i];
  int slot = atomicAdd(&fill[cid], 1);
  CellRec r;
  r.q[0] = qpos[3 * i];
  r.q[1] = qpos[3 * i + 1];
  r.q[2] = qpos[3 * i + 2];
  r.j = static_cast<int32_t>(i);
  r.pad = 0;
  rec[start[cid] + slot] = r;
}

// exclusive-to-inclusive prefix sum over the 64 lanes of a wave
__device__ inline int wave_inclusive_scan(int v) {
  const int lane = lane_id();
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int t = __shfl_up(v, off);
    if (lane >= off) v += t;
  }
  return v;
}

// The stencil of one centre as runs of bins: a run is the bins of one
// (axis-0, axis-1) offset whose axis-2 bins are consecutive with one image
// index, so its atoms are one contiguous range of the bin-ordered records.
struct SegLds {
  int64_t off[3][kMaxSeg];   // image displacement sum_b s_b Q(h_b) minus Q(r_i)
  int32_t begin[kMaxSeg];    // first record of the run
  int32_t vend[kMaxSeg];     // end of the run in the centre's list of candidates
  int32_t s[3][kMaxSeg];     // image indices of the run
};

// Visits every candidate (record, image) of the stencil of centre i and
// calls f(j, s0, s1, s2, pred) on chunks of 64 (one per lane, pred false on
// idle lanes); pred is the exact membership test with the centre itself
// (j = i, n = 0) excluded.  The image index of a pair is n = s - m_j + m_i
// with m the wrap counts of binning.  Wave-uniform control flow.
template <bool TRIC, class Fn>
__device__ inline void for_stencil(const GridDev& g, int64_t i, const int64_t* __restrict__ qpos,
                                   const int32_t* __restrict__ cell_of,
                                   const int32_t* __restrict__ start,
                                   const CellRec* __restrict__ rec, SegLds& sg, Fn&& f) {
  const int lane = lane_id();
  const int64_t qi0 = qpos[3 * i], qi1 = qpos[3 * i + 1], qi2 = qpos[3 * i + 2];
  const int cid_i = cell_of[i];
  const int ci0 = cid_i / (g.nc1 * g.nc2);
  const int ci1 = (cid_i / g.nc2) % g.nc1;
  const int ci2 = cid_i % g.nc2;
  const int lo2 = ci2 - g.re2, hi2 = ci2 + g.re2;
  const int s2lo = static_cast<int>(floor_div(lo2, g.nc2));
  const int nr = static_cast<int>(floor_div(hi2, g.nc2)) - s2lo + 1;   // image runs along axis 2
  const int n1 = 2 * g.re1 + 1;
  const int nseg = (2 * g.re0 + 1) * n1 * nr;
  for (int sb = 0; sb < nseg; sb += kMaxSeg) {
    const int q = sb + lane;
    int len = 0;
    if (q < nseg) {
      const int r = q % nr, p = q / nr;
      const int t0 = ci0 + p / n1 - g.re0, t1 = ci1 + p % n1 - g.re1;
      const int s0 = static_cast<int>(floor_div(t0, g.nc0));
      const int s1 = static_cast<int>(floor_div(t1, g.nc1));
      const int s2 = s2lo + r;
      const int w0 = t0 - s0 * g.nc0, w1 = t1 - s1 * g.nc1;
      const int a = max(lo2, s2 * g.nc2) - s2 * g.nc2;
      const int b = min(hi2, s2 * g.nc2 + g.nc2 - 1) - s2 * g.nc2;
      const int base = (w0 * g.nc1 + w1) * g.nc2;
      const int beg = start[base + a];
      len = start[base + b + 1] - beg;
      int64_t ox, oy, oz;
      if (!TRIC) {
        ox = s0 * g.qh[0] - qi0;
        oy = s1 * g.qh[4] - qi1;
        oz = s2 * g.qh[8] - qi2;
      } else {
        ox = s0 * g.qh[0] + s1 * g.qh[3] + s2 * g.qh[6] - qi0;
        oy = s0 * g.qh[1] + s1 * g.qh[4] + s2 * g.qh[7] - qi1;
        oz = s0 * g.qh[2] + s1 * g.qh[5] + s2 * g.qh[8] - qi2;
      }
      sg.off[0][lane] = ox;
      sg.off[1][lane] = oy;
      sg.off[2][lane] = oz;
      sg.begin[lane] = beg;
      sg.s[0][lane] = s0;
      sg.s[1][lane] = s1;
      sg.s[2][lane] = s2;
    }
    const int vend = wave_inclusive_scan(len);
    sg.vend[lane] = vend;
    const int total = __shfl(vend, kWave - 1);
    wave_local_sync();
    int seg = 0;   // the run of this lane's candidate (candidates advance, so does the run)
    for (int k0 = 0; k0 < total; k0 += kWave) {
      const int k = k0 + lane;
      bool pred = false;
      int32_t j = 0;
      int sx = 0, sy = 0, sz = 0;
      if (k < total) {
        while (sg.vend[seg] <= k) ++seg;
        const int first = seg > 0 ? sg.vend[seg - 1] : 0;
        const CellRec c = rec[sg.begin[seg] + (k - first)];
        j = c.j;
        sx = sg.s[0][seg];
        sy = sg.s[1][seg];
        sz = sg.s[2][seg];
        pred = within(c.q[0] + sg.off[0][seg], c.q[1] + sg.off[1][seg], c.q[2] + sg.off[2][seg],
                      g.rq) &&
               !(j == i && sx == 0 && sy == 0 && sz == 0);
      }
      f(j, sx, sy, sz, pred);
    }
    wave_local_sync();   // the next batch of runs overwrites the table
  }
}

template <bool TRIC>
__global__ void __launch_bounds__(kBlock) count_kernel(int64_t n, GridDev g,
                                                       const int64_t* __restrict__ qpos,
                                                       const int32_t* __restrict__ cell_of,
                                                       const int32_t* __restrict__ start,
                                                       const CellRec* __restrict__ rec,
                                                       int64_t* __restrict__ counts,
                                                       int64_t* __restrict__ flags) {
  __shared__ SegLds segs[kWavesPerBlock];
  SegLds& sg = segs[threadIdx.x / kWave];
  const int64_t nwaves = int64_t(gridDim.x) * kWavesPerBlock;
  int64_t longest = 0;
  for (int64_t i = xcd_block(blockIdx.x, gridDim.x) * kWavesPerBlock + threadIdx.x / kWave; i < n;
       i += nwaves) {
    int64_t total = 0;
    for_stencil<TRIC>(g, i, qpos, cell_of, start, rec, sg, [&](int32_t, int, int, int, bool pred) {
      total += __popcll(__ballot(pred));
    });
    if (lane_id() == 0) counts[i] = total;
    longest = total > longest ? total : longest;
  }
  if (lane_id() == 0 && longest > 0)
    atomicMax(reinterpret_cast<unsigned long long*>(flags + kFlagMaxRow),
              static_cast<unsigned long long>(longest));
}

// ---------------------------------------------------------------------------
// int64 exclusive scan: out[0..n] with out[n] = total
constexpr int kScanPer = 8;
constexpr int kScanTile = kBlock * kScanPer;

__device__ inline int64_t block_exclusive_scan(int64_t v, int64_t* sh, int64_t* total) {
  int t = threadIdx.x;
  sh[t] = v;
  __syncthreads();
  for (int off = 1; off < kBlock; off <<= 1) {
    int64_t add = t >= off ? sh[t - off] : 0;
    __syncthreads();
    sh[t] += add;
    __syncthreads();
  }
  int64_t incl = sh[t];
  *total = sh[kBlock - 1];
  __syncthreads();
  return incl - v;
}

template <class T>
__global__ void __launch_bounds__(kBlock) scan_partials_kernel(const T* __restrict__ in, int64_t n,
                                                               int64_t* __restrict__ partials) {
  __shared__ int64_t sh[kBlock];
  int64_t base = blockIdx.x * int64_t(kScanTile) + threadIdx.x * kScanPer;
  int64_t s = 0;
  for (int k = 0; k < kScanPer; ++k)
    if (base + k < n) s += in[base + k];
  int64_t tot;
  block_exclusive_scan(s, sh, &tot);
  if (threadIdx.x == 0) partials[blockIdx.x] = tot;
}

__global__ void __launch_bounds__(kBlock) scan_top_kernel(int64_t* __restrict__ partials,
                                                          int64_t nparts) {
  __shared__ int64_t sh[kBlock];
  int64_t carry = 0;
  for (int64_t b = 0; b < nparts; b += kBlock) {
    int64_t idx = b + threadIdx.x;
    int64_t v = idx < nparts ? partials[idx] : 0;
    int64_t tot;
    int64_t ex = block_exclusive_scan(v, sh, &tot);
    if (idx < nparts) partials[idx] = ex + carry;
    carry += tot;
  }
}

template <class T>
__global__ void __launch_bounds__(kBlock) scan_apply_kernel(const T* __restrict__ in, int64_t n,
                                                            const int64_t* __restrict__ partials,
                                                            T* __restrict__ out) {
  __shared__ int64_t sh[kBlock];
  int64_t base = blockIdx.x * int64_t(kScanTile) + threadIdx.x * kScanPer;
  int64_t v[kScanPer];
  int64_t s = 0;
  for (int k = 0; k < kScanPer; ++k) {
    v[k] = base + k < n ? int64_t(in[base + k]) : 0;
    s += v[k];
  }
  int64_t tot;
  int64_t run = block_exclusive_scan(s, sh, &tot) + partials[blockIdx.x];
  for (int k = 0; k < kScanPer; ++k) {
    if (base + k < n) out[base + k] = static_cast<T>(run);
    run += v[k];
  }
  if (base <= n - 1 && n - 1 < base + kScanPer) out[n] = static_cast<T>(run);  // thread holding the last element
}

// exclusive scan out[0..n] of in[0..n) with out[n] = the total (int32 or int64)
template <class T>
int exclusive_scan(const T* in, int64_t n, T* out, DevBuf& partials, hipStream_t st) {
  int64_t nb = (n + kScanTile - 1) / kScanTile;
  if (nb == 0) nb = 1;
  DPA4C_TRY(partials.ensure(sizeof(int64_t) * nb));
  hipLaunchKernelGGL(scan_partials_kernel<T>, dim3(nb), dim3(kBlock), 0, st, in, n,
                     partials.as<int64_t>());
  hipLaunchKernelGGL(scan_top_kernel, dim3(1), dim3(kBlock), 0, st, partials.as<int64_t>(), nb);
  hipLaunchKernelGGL(scan_apply_kernel<T>, dim3(nb), dim3(kBlock), 0, st, in, n,
                     partials.as<int64_t>(), out);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

// ---------------------------------------------------------------------------
// Canonical key of a list entry: rows are sorted by it.
__device__ inline int64_t entry_key(int32_t j, int32_t sh) {
  return (int64_t(j) << 24) | int64_t(sh & 0xFFFFFF);
}

// Writes the keys kb[0, len) of a row at their ranks, the number of smaller
// keys in the row (keys of a row are distinct), PER keys per lane at a time
// against one broadcast read of every key; with ``jsamp`` also j of every
// entry at an absolute position 16 g, to jsamp[g].
template <int PER, class KB>
__device__ __forceinline__ void rank_row(int len, int64_t r0, KB* kb, int32_t* __restrict__ nbr_j,
                                         int32_t* __restrict__ nbr_shift,
                                         int32_t* __restrict__ jsamp) {
  const int lane = lane_id();
  for (int t0 = 0; t0 < len; t0 += kWave * PER) {
    int64_t mine[PER];
    int rank[PER];
#pragma unroll
    for (int r = 0; r < PER; ++r) {
      const int t = t0 + lane + kWave * r;
      mine[r] = t < len ? kb[t] : INT64_MAX;
      rank[r] = 0;
    }
    for (int u = 0; u < len; ++u) {
      const int64_t ku = kb[u];
#pragma unroll
      for (int r = 0; r < PER; ++r) rank[r] += ku < mine[r] ? 1 : 0;
    }
#pragma unroll
    for (int r = 0; r < PER; ++r) {
      const int t = t0 + lane + kWave * r;
      if (t < len) {
        const int64_t at = r0 + rank[r];
        const int32_t j = static_cast<int32_t>(mine[r] >> 24);
        nbr_j[at] = j;
        nbr_shift[at] = static_cast<int32_t>(mine[r] & 0xFFFFFF);
        if (jsamp && (at & 15) == 0) jsamp[at >> 4] = j;
      }
    }
  }
}

typedef long long i64x2 __attribute__((ext_vector_type(2)));

// The same ranks for a row held in LDS, counted inside buckets: the keys
// are grouped by j into at most 64 buckets of one power-of-two width over
// the row's range of j, so a key's bucket never decreases as the key grows
// and its rank is the number of keys in lower buckets plus the number of
// smaller keys in its own bucket.  The keys are regrouped in place by bucket
// (in any order inside one); each lane then takes grouped keys and compares
// only with its bucket.  ``boff`` and ``bend`` are 64 ints of the wave's LDS;
// kb (16-byte aligned) has room for kRankBlock keys past the row.
template <int PER, class KB>
__device__ __forceinline__ void rank_row_lds(int len, int64_t r0, KB* kb, int32_t* boff,
                                             int32_t* bend, int32_t* __restrict__ nbr_j,
                                             int32_t* __restrict__ nbr_shift,
                                             int32_t* __restrict__ jsamp) {
  const int lane = lane_id();
  int64_t key[PER];
  int32_t jlo = INT32_MAX, jhi = INT32_MIN;
#pragma unroll
  for (int r = 0; r < PER; ++r) {
    const int t = lane + kWave * r;
    key[r] = t < len ? kb[t] : 0;
    if (t < len) {
      const int32_t j = static_cast<int32_t>(key[r] >> 24);
      jlo = j < jlo ? j : jlo;
      jhi = j > jhi ? j : jhi;
    }
  }
#pragma unroll
  for (int off = kWave / 2; off >= 1; off >>= 1) {
    const int32_t lo = __shfl_xor(jlo, off), hi = __shfl_xor(jhi, off);
    jlo = lo < jlo ? lo : jlo;
    jhi = hi > jhi ? hi : jhi;
  }
  jlo = __builtin_amdgcn_readfirstlane(jlo);
  jhi = __builtin_amdgcn_readfirstlane(jhi);
  // width 2^sh with (jhi - jlo) >> sh < 64
  const uint32_t span = static_cast<uint32_t>(jhi - jlo);
  const int sh = span < 64u ? 0 : 26 - __clz(span);
  auto bucket = [&](int64_t k) {
    return static_cast<int>(static_cast<uint32_t>(static_cast<int32_t>(k >> 24) - jlo) >> sh);
  };
  boff[lane] = 0;
  wave_local_sync();
  int bk[PER], slot[PER];
#pragma unroll
  for (int r = 0; r < PER; ++r) {
    bk[r] = 0;
    slot[r] = 0;
    if (lane + kWave * r < len) {
      bk[r] = bucket(key[r]);
      slot[r] = atomicAdd(&boff[bk[r]], 1);
    }
  }
  wave_local_sync();
  const int cnt = boff[lane];
  const int incl = wave_inclusive_scan(cnt);
  wave_local_sync();
  boff[lane] = incl - cnt;
  bend[lane] = incl;
  wave_local_sync();
#pragma unroll
  for (int r = 0; r < PER; ++r)
    if (lane + kWave * r < len) kb[boff[bk[r]] + slot[r]] = key[r];
  if (lane < kRankBlock) kb[len + lane] = INT64_MAX;   // sentinels past the row
  wave_local_sync();
  // Every key before a bucket is smaller than the bucket's keys and every
  // key after it larger (or a sentinel), so a key's rank is counted over
  // whole aligned blocks of kRankBlock keys around its bucket.
#pragma unroll
  for (int r = 0; r < PER; ++r) {
    const int t = lane + kWave * r;
    if (t < len) {
      const int64_t k = kb[t];
      const int b = bucket(k);
      const int lo = boff[b] & ~(kRankBlock - 1), hi = bend[b];
      int rank = lo;
      for (int u = lo; u < hi; u += kRankBlock) {
        const i64x2* q = reinterpret_cast<const i64x2*>(kb + u);
#pragma unroll
        for (int v = 0; v < kRankBlock / 2; ++v) {
          const i64x2 x = q[v];
          rank += (x.x < k ? 1 : 0) + (x.y < k ? 1 : 0);
        }
      }
      const int64_t at = r0 + rank;
      const int32_t j = static_cast<int32_t>(k >> 24);
      nbr_j[at] = j;
      nbr_shift[at] = static_cast<int32_t>(k & 0xFFFFFF);
      if (jsamp && (at & 15) == 0) jsamp[at >> 4] = j;
    }
  }
}

// One row: the accepted keys into kb[0, len) in candidate order, then
// each written at its rank.  ``kb`` is the wave's LDS row (LDS_ROW) or, for
// a row longer than kMaxRow, a global scratch row (inlined for each, so LDS
// rows use LDS instructions).
template <bool TRIC, bool LDS_ROW, class KB>
__device__ __forceinline__ void fill_row(const GridDev& g, int64_t i, int64_t r0, int len, KB* kb,
                                         const int64_t* __restrict__ qpos,
                                         const int32_t* __restrict__ wrap,
                                         const int32_t* __restrict__ cell_of,
                                         const int32_t* __restrict__ start,
                                         const CellRec* __restrict__ rec, SegLds& sg,
                                         int32_t* __restrict__ nbr_j,
                                         int32_t* __restrict__ nbr_shift,
                                         int32_t* __restrict__ jsamp, int64_t* __restrict__ flags) {
  const int mi0 = wrap[3 * i], mi1 = wrap[3 * i + 1], mi2 = wrap[3 * i + 2];
  int fill = 0;
  bool shift_bad = false;
  for_stencil<TRIC>(g, i, qpos, cell_of, start, rec, sg, [&](int32_t j, int s0, int s1, int s2,
                                                             bool pred) {
    uint64_t m;
    const int pre = ballot_prefix(pred, &m);
    if (pred) {
      const int nx = s0 - wrap[3 * j] + mi0;
      const int ny = s1 - wrap[3 * j + 1] + mi1;
      const int nz = s2 - wrap[3 * j + 2] + mi2;
      if (nx < -127 || nx > 127 || ny < -127 || ny > 127 || nz < -127 || nz > 127) shift_bad = true;
      const int slot = fill + pre;
      if (slot < len) kb[slot] = entry_key(j, pack_shift(nx, ny, nz));
    }
    fill += __popcll(m);
  });
  if (shift_bad)
    atomicOr(reinterpret_cast<unsigned long long*>(flags), (unsigned long long)kFlagShift);
  if constexpr (LDS_ROW) {
    wave_local_sync();
    if (len <= kWave) rank_row<1>(len, r0, kb, nbr_j, nbr_shift, jsamp);
    else if (len <= 2 * kWave) rank_row_lds<2>(len, r0, kb, sg.begin, sg.vend, nbr_j, nbr_shift, jsamp);
    else if (len <= 4 * kWave) rank_row_lds<4>(len, r0, kb, sg.begin, sg.vend, nbr_j, nbr_shift, jsamp);
    else rank_row_lds<8>(len, r0, kb, sg.begin, sg.vend, nbr_j, nbr_shift, jsamp);
    wave_local_sync();   // the row's keys are read before the next row overwrites them
  } else {
    wave_lds_sync();     // the keys are global memory here: the stores are waited for
    if (len <= kWave) rank_row<1>(len, r0, kb, nbr_j, nbr_shift, jsamp);
    else if (len <= 2 * kWave) rank_row<2>(len, r0, kb, nbr_j, nbr_shift, jsamp);
    else if (len <= 4 * kWave) rank_row<4>(len, r0, kb, nbr_j, nbr_shift, jsamp);
    else rank_row<8>(len, r0, kb, nbr_j, nbr_shift, jsamp);
    wave_lds_sync();
  }
}

// Rows of the skin list: the accepted candidates of centre i as keys
// (j, packed n), each written at its rank in the row, so rows come out in
// canonical order.  With ``jsamp`` the neighbour index of every entry at an
// absolute position 16 g also goes to jsamp[g], for the reverse search.
// Rows longer than kMaxRow collect their keys in long_keys[row_ptr[i] ...]
// instead of LDS (the host passes it when the count found such rows;
// without it they are flagged).
template <bool TRIC>
__global__ void __launch_bounds__(kBlock) fill_kernel(int64_t n, GridDev g,
                                                      const int64_t* __restrict__ qpos,
                                                      const int32_t* __restrict__ wrap,
                                                      const int32_t* __restrict__ cell_of,
                                                      const int32_t* __restrict__ start,
                                                      const CellRec* __restrict__ rec,
                                                      const int64_t* __restrict__ row_ptr,
                                                      int32_t* __restrict__ nbr_j,
                                                      int32_t* __restrict__ nbr_shift, int64_t cap,
                                                      int32_t* __restrict__ jsamp,
                                                      int64_t* __restrict__ long_keys,
                                                      int64_t* __restrict__ flags) {
  __shared__ SegLds segs[kWavesPerBlock];
  __shared__ alignas(16) int64_t keys_all[kWavesPerBlock][kMaxRow + kRankBlock];
  if (row_ptr[n] > cap) {
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      atomicOr(reinterpret_cast<unsigned long long*>(flags), (unsigned long long)kFlagCapacity);
      atomicMax(reinterpret_cast<unsigned long long*>(flags + 2), (unsigned long long)row_ptr[n]);
    }
    return;
  }
  const int w = threadIdx.x / kWave;
  SegLds& sg = segs[w];
  const int64_t nwaves = int64_t(gridDim.x) * kWavesPerBlock;
  for (int64_t i = xcd_block(blockIdx.x, gridDim.x) * kWavesPerBlock + w; i < n; i += nwaves) {
    const int64_t r0 = row_ptr[i];
    const int len = static_cast<int>(row_ptr[i + 1] - r0);
    if (len <= kMaxRow) {
      fill_row<TRIC, true>(g, i, r0, len, keys_all[w], qpos, wrap, cell_of, start, rec, sg, nbr_j,
                     nbr_shift, jsamp, flags);
    } else if (long_keys) {
      fill_row<TRIC, false>(g, i, r0, len, long_keys + r0, qpos, wrap, cell_of, start, rec, sg, nbr_j,
                     nbr_shift, jsamp, flags);
    } else if (lane_id() == 0) {
      atomicOr(reinterpret_cast<unsigned long long*>(flags), (unsigned long long)kFlagRowTooLong);
    }
  }
}

// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(kBlock) fill_i64_kernel(int64_t* __restrict__ p, int64_t n,
                                                          int64_t v) {
  for (int64_t i = blockIdx.x * int64_t(kBlock) + threadIdx.x; i < n; i += int64_t(gridDim.x) * kBlock)
    p[i] = v;
}

// jsamp[g] = nbr_j[16 g], for a list built elsewhere (a caller's)
__global__ void __launch_bounds__(kBlock) jsamp_kernel(const int64_t* __restrict__ row_ptr, int64_t n,
                                                       const int32_t* __restrict__ nbr_j, int64_t cap,
                                                       int32_t* __restrict__ jsamp) {
  int64_t total = row_ptr[n];
  total = total < cap ? (total < 0 ? 0 : total) : cap;
  for (int64_t g = blockIdx.x * int64_t(kBlock) + threadIdx.x; 16 * g < total;
       g += int64_t(gridDim.x) * kBlock)
    jsamp[g] = nbr_j[16 * g];
}

// A row outside [0, cap] (a malformed caller list) gets no reverse entries and
// is nobody's reverse row, like the compaction, which keeps nothing of it.
__device__ inline bool row_ok(int64_t b, int64_t e, int64_t cap) { return b >= 0 && e >= b && e <= cap; }

// The reverse search of entry s = (i -> j, n): the position of the entry
// (i, -n) of row j, written to rev[s], and s to rev of that entry (both
// positions in the whole list).  Row j is ordered by neighbour index,
// so the entries (i, m) of row j are consecutive and begin at the first
// entry with neighbour index >= i: the samples of row j (the neighbour
// index at every absolute position 16 g inside it) are bisected for the
// aligned block of 16 entries that holds it, that block is compared at once
// (four 16-byte loads with VEC, one load per entry without), and the entries
// (i, m) from there are matched on the image.
template <bool VEC>
__device__ inline bool reverse_search(int64_t n, int32_t i, int64_t s, int32_t j, int32_t sh,
                                      const int64_t* __restrict__ row_ptr,
                                      const int32_t* __restrict__ nbr_j,
                                      const int32_t* __restrict__ nbr_shift, int64_t cap,
                                      const int32_t* __restrict__ jsamp,
                                      int64_t* __restrict__ rev) {
  const int32_t want_sh = negate_shift(sh);
  if (j < 0 || j >= n) return false;
  const int64_t jb = row_ptr[j], je = row_ptr[j + 1];
  if (!row_ok(jb, je, cap) || je == jb) return false;
  const int64_t g0 = (jb + 15) >> 4, g1 = (je - 1) >> 4;   // samples inside the row
  int64_t l = g0;                                           // first sample >= i
  if (g0 <= g1) {
    int64_t h = g1 + 1;
    while (l < h) {
      const int64_t m = (l + h) >> 1;
      if (jsamp[m] < i) l = m + 1;
      else h = m;
    }
  }
  // the first entry >= i lies in [lo, hi), inside the aligned block [16 q, 16 q + 16)
  const int64_t lo = l > g0 ? 16 * (l - 1) : jb;
  const int64_t hi = l <= g1 ? 16 * l : je;
  const int64_t q16 = l > g0 ? 16 * (l - 1) : 16 * (g0 - 1);
  int64_t p = lo;
  if (VEC) {
    const int4* blk = reinterpret_cast<const int4*>(nbr_j + q16);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int64_t t = q16 + 4 * v;
      if (t + 3 >= lo && t < hi) {
        const int4 x = blk[v];
        p += (t >= lo && t < hi && x.x < i) + (t + 1 >= lo && t + 1 < hi && x.y < i) +
             (t + 2 >= lo && t + 2 < hi && x.z < i) + (t + 3 >= lo && t + 3 < hi && x.w < i);
      }
    }
  } else {
#pragma unroll
    for (int t = 0; t < 16; ++t)
      if (lo + t < hi && nbr_j[lo + t] < i) ++p;
  }
  for (int64_t t = p; t < je && nbr_j[t] == i; ++t)
    if (nbr_shift[t] == want_sh) {
      rev[s] = t;
      rev[t] = s;
      return true;
    }
  return false;
}

// skin_rev[s] = position in the list of the reverse of entry s (i -> j, n),
// the entry (i, -n) of row j, or -1.  A symmetric list pairs every entry with its
// reverse, so only the canonical entry of a pair, the one with
// key(j, n) > key(i, -n) (that is j > i, or a periodic self image with the
// larger shift), searches and writes both indices.  One wave takes rows in
// turn and queues their canonical entries in LDS, so every search round
// runs 64 searches.  Entries whose partner is missing (a malformed caller
// list) keep the -1 of the fill before.  With ``paired`` the pairs found
// are counted (one atomic per wave), so the caller can tell a symmetric list
// (2 x pairs = entries) from one that is not.  With ``order`` (the
// neighbour build's atom records in bin order) the rows are taken in that
// spatial order, so that centres searched close in time share their rows j
// in L2; the results do not depend on the order.
template <bool VEC>
__global__ void __launch_bounds__(kBlock) skin_rev_kernel(int64_t n, const int64_t* __restrict__ row_ptr,
                                                          const int32_t* __restrict__ nbr_j,
                                                          const int32_t* __restrict__ nbr_shift,
                                                          int64_t cap,
                                                          const int32_t* __restrict__ jsamp,
                                                          int64_t* __restrict__ rev,
                                                          unsigned long long* __restrict__ paired,
                                                          const CellRec* __restrict__ order) {
  __shared__ int64_t qs_all[kWavesPerBlock][2 * kWave];
  __shared__ int32_t qi_all[kWavesPerBlock][2 * kWave];
  __shared__ int32_t qj_all[kWavesPerBlock][2 * kWave];   // (j, n) of each queued entry
  __shared__ int32_t qh_all[kWavesPerBlock][2 * kWave];
  const int w = threadIdx.x / kWave;
  int64_t* qs = qs_all[w];
  int32_t* qi = qi_all[w];
  int32_t* qj = qj_all[w];
  int32_t* qh = qh_all[w];
  const int64_t nwaves = int64_t(gridDim.x) * kWavesPerBlock;
  const int lane = lane_id();
  unsigned long long found = 0;
  int qn = 0;   // queued searches (wave-uniform)
  // runs the first ``count`` (<= 64) queued searches and moves the rest down
  auto run = [&](int count) {
    const bool hit = lane < count &&
                     reverse_search<VEC>(n, qi[lane], qs[lane], qj[lane], qh[lane], row_ptr, nbr_j,
                                         nbr_shift, cap,
                                         jsamp, rev);
    found += __popcll(__ballot(hit));
    const int rest = qn - count;
    int64_t ks = 0;
    int32_t ki = 0, kj = 0, kh = 0;
    if (lane < rest) {
      ks = qs[count + lane];
      ki = qi[count + lane];
      kj = qj[count + lane];
      kh = qh[count + lane];
    }
    wave_local_sync();
    if (lane < rest) {
      qs[lane] = ks;
      qi[lane] = ki;
      qj[lane] = kj;
      qh[lane] = kh;
    }
    wave_local_sync();
    qn = rest;
  };
  for (int64_t r = xcd_block(blockIdx.x, gridDim.x) * kWavesPerBlock + w; r < n; r += nwaves) {
    const int64_t i = order ? order[r].j : r;
    const int64_t b = row_ptr[i], e = row_ptr[i + 1];
    if (!row_ok(b, e, cap)) continue;
    for (int64_t s0 = b; s0 < e; s0 += kWave) {
      const int64_t s = s0 + lane;
      bool canon = false;
      int32_t j = 0, sh = 0;
      if (s < e) {
        j = nbr_j[s];
        sh = nbr_shift[s];
        canon = entry_key(j, sh) > entry_key(static_cast<int32_t>(i), negate_shift(sh));
      }
      uint64_t m;
      const int pre = ballot_prefix(canon, &m);
      if (canon) {
        qs[qn + pre] = s;
        qi[qn + pre] = static_cast<int32_t>(i);
        qj[qn + pre] = j;
        qh[qn + pre] = sh;
      }
      qn += __popcll(m);
      wave_local_sync();
      if (qn >= kWave) run(kWave);
    }
  }
  if (qn > 0) run(qn);
  if (paired && lane == 0 && found) atomicAdd(paired, found);
}

// per-axis minimum and maximum of the fixed-point positions (exact integer
// min/max, so independent of the order of the atomics); out = [min x, y, z,
// max x, y, z], initialised by the caller to (INT64_MAX, INT64_MIN)
__global__ void __launch_bounds__(kBlock) extent_kernel(const double* __restrict__ pos, int64_t n,
                                                        long long* __restrict__ out) {
  __shared__ long long sh[6][kWavesPerBlock];
  long long lo[3] = {INT64_MAX, INT64_MAX, INT64_MAX}, hi[3] = {INT64_MIN, INT64_MIN, INT64_MIN};
  for (int64_t i = blockIdx.x * int64_t(kBlock) + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * kBlock) {
    for (int a = 0; a < 3; ++a) {
      const double x = pos[3 * i + a];
      if (!isfinite(x) || fabs(x) > 1.0e12) continue;   // flagged by the build
      const long long q = qfix(x);
      lo[a] = q < lo[a] ? q : lo[a];
      hi[a] = q > hi[a] ? q : hi[a];
    }
  }
  for (int off = 1; off < kWave; off <<= 1)
    for (int a = 0; a < 3; ++a) {
      const long long l = __shfl_xor(lo[a], off), h = __shfl_xor(hi[a], off);
      lo[a] = l < lo[a] ? l : lo[a];
      hi[a] = h > hi[a] ? h : hi[a];
    }
  const int w = threadIdx.x / kWave;
  if (lane_id() == 0)
    for (int a = 0; a < 3; ++a) {
      sh[a][w] = lo[a];
      sh[3 + a][w] = hi[a];
    }
  __syncthreads();
  if (threadIdx.x < 6) {
    const int a = threadIdx.x;
    long long v = sh[a][0];
    for (int k = 1; k < kWavesPerBlock; ++k) v = a < 3 ? (sh[a][k] < v ? sh[a][k] : v)
                                                       : (sh[a][k] > v ? sh[a][k] : v);
    if (a < 3) atomicMin(out + a, v);
    else atomicMax(out + a, v);
  }
}

__global__ void extent_init_kernel(long long* out) {
  if (threadIdx.x < 6) out[threadIdx.x] = threadIdx.x < 3 ? INT64_MAX : INT64_MIN;
}

int waves_grid(int64_t n) {
  int64_t blocks = (n + kWavesPerBlock - 1) / kWavesPerBlock;
  if (blocks > 4096) blocks = 4096;
  return static_cast<int>(blocks < 1 ? 1 : blocks);
}

}  // namespace

int make_grid(const double cell[9], int64_t rq, CellGrid* g) {
  if (rq <= 0 || rq > int64_t(1000) * int64_t(kQScale)) {
    set_error("bad neighbour radius");
    return DPA4C_ERR_INVALID_ARG;
  }
  for (int k = 0; k < 9; ++k)
    if (!std::isfinite(cell[k]) || std::fabs(cell[k]) > 1.0e6) {
      set_error("cell entries must be finite and below 1e6 A");
      return DPA4C_ERR_INVALID_ARG;
    }
  g->rq = rq;
  g->ncell = 1;
  g->tric = 0;
  for (int a = 0; a < 3; ++a)
    for (int b = 0; b < 3; ++b)
      if (a != b && cell[3 * a + b] != 0.0) g->tric = 1;
  for (int k = 0; k < 9; ++k) {
    g->h[k] = cell[k];
    g->qh[k] = static_cast<int64_t>(std::rint(cell[k] * kQScale));
  }
  // inverse lattice matrix (rows of ``cell`` are the lattice vectors)
  const double* h = cell;
  const double det = h[0] * (h[4] * h[8] - h[5] * h[7]) - h[1] * (h[3] * h[8] - h[5] * h[6]) +
                     h[2] * (h[3] * h[7] - h[4] * h[6]);
  if (!g->tric) {
    for (int a = 0; a < 3; ++a)
      if (!(cell[4 * a] > 0)) {
        set_error("the diagonal of an orthorhombic cell must be positive");
        return DPA4C_ERR_INVALID_ARG;
      }
  }
  double vol = std::fabs(det);
  double hmax = 0.0;
  for (int k = 0; k < 9; ++k) hmax = std::max(hmax, std::fabs(cell[k]));
  if (!(vol > 1e-9 * hmax * hmax * hmax) || !(vol > 0)) {
    set_error("the cell is singular");
    return DPA4C_ERR_INVALID_ARG;
  }
  const double cof[9] = {h[4] * h[8] - h[5] * h[7], h[2] * h[7] - h[1] * h[8],
                         h[1] * h[5] - h[2] * h[4], h[5] * h[6] - h[3] * h[8],
                         h[0] * h[8] - h[2] * h[6], h[2] * h[3] - h[0] * h[5],
                         h[3] * h[7] - h[4] * h[6], h[1] * h[6] - h[0] * h[7],
                         h[0] * h[4] - h[1] * h[3]};
  for (int k = 0; k < 9; ++k) g->inv[k] = cof[k] / det;
  const double r = double(rq) / kQScale;
  // bins of about half the radius (sub = 2 per radius, stencil reach 2); a
  // grid of more than kMaxFineBins bins (a sparse system in a large cell)
  // falls back to radius-wide bins
  constexpr int64_t kMaxFineBins = int64_t(1) << 24;
  for (int sub = 2; sub >= 1; --sub) {
    g->ncell = 1;
    for (int a = 0; a < 3; ++a) {
      int64_t nc;
      if (!g->tric) {
        const int64_t L = g->qh[4 * a];
        nc = sub * L / g->rq;
        if (nc < 1) nc = 1;
        if (nc > 1024) nc = 1024;
        g->reach[a] = static_cast<int>((g->rq * nc + L - 1) / L);
      } else {
        // distance between the lattice planes of axis a: V / |h_b x h_c|
        const double* u = h + 3 * ((a + 1) % 3);
        const double* v = h + 3 * ((a + 2) % 3);
        const double cx = u[1] * v[2] - u[2] * v[1], cy = u[2] * v[0] - u[0] * v[2],
                     cz = u[0] * v[1] - u[1] * v[0];
        const double d = vol / std::sqrt(cx * cx + cy * cy + cz * cz);
        nc = static_cast<int64_t>(std::floor(sub * d / r));
        if (nc < 1) nc = 1;
        if (nc > 1024) nc = 1024;
        const double re = std::ceil((r + 1e-6) * double(nc) / d);
        if (re > 1024.0) {
          set_error("the cell is too thin for the neighbour radius");
          return DPA4C_ERR_UNSUPPORTED;
        }
        g->reach[a] = static_cast<int>(re);
      }
      g->nc[a] = static_cast<int>(nc);
      g->ncell *= nc;
    }
    if (g->ncell <= kMaxFineBins) break;
  }
  return 0;
}

int ensure_scratch(NeighborScratch& nb, int64_t n, const CellGrid& g) {
  DPA4C_TRY(nb.qpos.ensure(sizeof(int64_t) * 3 * n));
  DPA4C_TRY(nb.wrap.ensure(sizeof(int32_t) * 3 * n));
  DPA4C_TRY(nb.cell_of.ensure(sizeof(int32_t) * n));
  DPA4C_TRY(nb.cell_cnt.ensure(sizeof(int32_t) * g.ncell));
  DPA4C_TRY(nb.cell_start.ensure(sizeof(int32_t) * (g.ncell + 1)));
  DPA4C_TRY(nb.cell_fill.ensure(sizeof(int32_t) * g.ncell));
  DPA4C_TRY(nb.cell_rec.ensure(sizeof(CellRec) * n));
  DPA4C_TRY(nb.counts.ensure(sizeof(int64_t) * n));
  // the bin counts and the row counts are scanned with the same partials
  const int64_t most = std::max<int64_t>(n, g.ncell);
  DPA4C_TRY(nb.partials.ensure(sizeof(int64_t) * size_t((most + kScanTile - 1) / kScanTile + 1)));
  return 0;
}

int build_skin_list(NeighborScratch& nb, const double* pos, int64_t n, const CellGrid& g,
                    int64_t* row_ptr, int64_t* flags, hipStream_t st) {
  int rc = ensure_scratch(nb, n, g);
  if (rc) return rc;
  GridDev gd = to_dev(g);
  int blocks = static_cast<int>((n + kBlock - 1) / kBlock);
  int cblocks = static_cast<int>((g.ncell + kBlock - 1) / kBlock);
  hipLaunchKernelGGL(zero_i32_kernel, dim3(cblocks), dim3(kBlock), 0, st,
                     nb.cell_cnt.as<int32_t>(), g.ncell);
  if (g.tric)
    hipLaunchKernelGGL(bin_kernel<true>, dim3(blocks), dim3(kBlock), 0, st, pos, n, gd,
                       nb.qpos.as<int64_t>(), nb.wrap.as<int32_t>(), nb.cell_of.as<int32_t>(),
                       nb.cell_cnt.as<int32_t>(), flags);
  else
    hipLaunchKernelGGL(bin_kernel<false>, dim3(blocks), dim3(kBlock), 0, st, pos, n, gd,
                       nb.qpos.as<int64_t>(), nb.wrap.as<int32_t>(), nb.cell_of.as<int32_t>(),
                       nb.cell_cnt.as<int32_t>(), flags);
  rc = exclusive_scan(nb.cell_cnt.as<int32_t>(), g.ncell, nb.cell_start.as<int32_t>(), nb.partials,
                      st);
  if (rc) return rc;
  hipLaunchKernelGGL(zero_i32_kernel, dim3(cblocks), dim3(kBlock), 0, st,
                     nb.cell_fill.as<int32_t>(), g.ncell);
  hipLaunchKernelGGL(place_kernel, dim3(blocks), dim3(kBlock), 0, st, n, nb.cell_of.as<int32_t>(),
                     nb.qpos.as<int64_t>(), nb.cell_start.as<int32_t>(),
                     nb.cell_fill.as<int32_t>(), nb.cell_rec.as<CellRec>());
  if (g.tric)
    hipLaunchKernelGGL(count_kernel<true>, dim3(waves_grid(n)), dim3(kBlock), 0, st, n, gd,
                       nb.qpos.as<int64_t>(), nb.cell_of.as<int32_t>(),
                       nb.cell_start.as<int32_t>(), nb.cell_rec.as<CellRec>(),
                       nb.counts.as<int64_t>(), flags);
  else
    hipLaunchKernelGGL(count_kernel<false>, dim3(waves_grid(n)), dim3(kBlock), 0, st, n, gd,
                       nb.qpos.as<int64_t>(), nb.cell_of.as<int32_t>(),
                       nb.cell_start.as<int32_t>(), nb.cell_rec.as<CellRec>(),
                       nb.counts.as<int64_t>(), flags);
  DPA4C_HIP_TRY(hipGetLastError());
  return exclusive_scan(nb.counts.as<int64_t>(), n, row_ptr, nb.partials, st);
}

int fill_skin_list(NeighborScratch& nb, int64_t n, const CellGrid& g, const int64_t* row_ptr,
                   int32_t* nbr_j, int32_t* nbr_shift, int64_t cap, int64_t* flags,
                   int64_t max_row, int32_t* jsamp, hipStream_t st) {
  GridDev gd = to_dev(g);
  int64_t* long_keys = nullptr;
  if (max_row > kMaxRow) {
    DPA4C_TRY(nb.long_keys.ensure(sizeof(int64_t) * size_t(cap < 1 ? 1 : cap)));
    long_keys = nb.long_keys.as<int64_t>();
  }
  if (g.tric)
    hipLaunchKernelGGL(fill_kernel<true>, dim3(waves_grid(n)), dim3(kBlock), 0, st, n, gd,
                       nb.qpos.as<int64_t>(), nb.wrap.as<int32_t>(), nb.cell_of.as<int32_t>(),
                       nb.cell_start.as<int32_t>(), nb.cell_rec.as<CellRec>(), row_ptr, nbr_j,
                       nbr_shift, cap, jsamp, long_keys, flags);
  else
    hipLaunchKernelGGL(fill_kernel<false>, dim3(waves_grid(n)), dim3(kBlock), 0, st, n, gd,
                       nb.qpos.as<int64_t>(), nb.wrap.as<int32_t>(), nb.cell_of.as<int32_t>(),
                       nb.cell_start.as<int32_t>(), nb.cell_rec.as<CellRec>(), row_ptr, nbr_j,
                       nbr_shift, cap, jsamp, long_keys, flags);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

int position_extent(const double* pos, int64_t n, int64_t* dev6, int64_t* host6, hipStream_t st) {
  long long* d = reinterpret_cast<long long*>(dev6);
  hipLaunchKernelGGL(extent_init_kernel, dim3(1), dim3(64), 0, st, d);
  int64_t blocks = (n + kBlock - 1) / kBlock;
  if (blocks > 1024) blocks = 1024;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(extent_kernel, dim3(blocks), dim3(kBlock), 0, st, pos, n, d);
  DPA4C_HIP_TRY(hipGetLastError());
  DPA4C_HIP_TRY(hipMemcpyAsync(host6, dev6, 6 * sizeof(int64_t), hipMemcpyDeviceToHost, st));
  DPA4C_HIP_TRY(hipStreamSynchronize(st));
  return 0;
}

int launch_skin_rev(const int64_t* row_ptr, const int32_t* nbr_j, const int32_t* nbr_shift,
                    int64_t n, int64_t cap, int32_t* jsamp, bool jsamp_ready, int64_t* skin_rev,
                    int64_t* paired, const NeighborScratch* order_of, hipStream_t st) {
  const CellRec* order = order_of ? order_of->cell_rec.as<CellRec>() : nullptr;
  if (n <= 0) return 0;
  int64_t sb = (cap + kBlock - 1) / kBlock;
  sb = sb < 1 ? 1 : (sb > 8192 ? 8192 : sb);
  if (!jsamp_ready) {
    int64_t jb = (cap / 16 + kBlock) / kBlock;
    jb = jb < 1 ? 1 : (jb > 4096 ? 4096 : jb);
    hipLaunchKernelGGL(jsamp_kernel, dim3(static_cast<unsigned>(jb)), dim3(kBlock), 0, st, row_ptr,
                       n, nbr_j, cap, jsamp);
  }
  hipLaunchKernelGGL(fill_i64_kernel, dim3(static_cast<unsigned>(sb)), dim3(kBlock), 0, st,
                     skin_rev, cap, int64_t(-1));
  // the block compare reads 16-byte groups of nbr_j: a list that is not
  // 16-byte aligned takes one load per entry
  const bool vec = (reinterpret_cast<uintptr_t>(nbr_j) & 15) == 0;
  if (vec)
    hipLaunchKernelGGL(skin_rev_kernel<true>, dim3(waves_grid(n)), dim3(kBlock), 0, st, n, row_ptr,
                       nbr_j, nbr_shift, cap, jsamp, skin_rev,
                       reinterpret_cast<unsigned long long*>(paired), order);
  else
    hipLaunchKernelGGL(skin_rev_kernel<false>, dim3(waves_grid(n)), dim3(kBlock), 0, st, n, row_ptr,
                       nbr_j, nbr_shift, cap, jsamp, skin_rev,
                       reinterpret_cast<unsigned long long*>(paired), order);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

}  // namespace dpa4c
