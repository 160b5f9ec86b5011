// Internal definitions shared by the HIP sources of the DPA4C library.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <type_traits>

namespace dpa4c {

constexpr double kEps = 1.0e-7;          // Eq. (edge-geometry) regulariser
constexpr double kQScale = 1048576.0;    // 2^20: fixed-point resolution of positions
constexpr int kWave = 64;

// Workgroups are handed to the 8 XCDs of the chip in turn (dispatch index b
// runs on XCD b % 8), and each XCD has its own L2.  xcd_block maps b to a
// work index so that every XCD takes one contiguous eighth of [0, nblocks):
// kernels whose rows gather the data of neighbouring atoms (positions,
// reverse rows, reverse gradients) then find most of it in their own L2.  A
// bijection on [0, nblocks).
__device__ inline int64_t xcd_block(int64_t b, int64_t nblocks) {
  constexpr int64_t kXcd = 8;
  const int64_t per = nblocks / kXcd, rem = nblocks % kXcd;
  const int64_t x = b % kXcd, k = b / kXcd;
  return x * per + (x < rem ? x : rem) + k;
}

// ---------------------------------------------------------------------------
// Compile-time profile (C0, L, R): every width of the model follows from it
// (Eqs. (degree-channels), (probe-ranks), (moment-width), (dim-out)).
// ---------------------------------------------------------------------------
constexpr int ceil_log2(int x) { return x <= 1 ? 0 : 1 + ceil_log2((x + 1) / 2); }
constexpr int imax(int a, int b) { return a > b ? a : b; }

template <int C0_, int L_, int R_>
struct Profile {
  static constexpr int C0 = C0_, L = L_, R = R_;
  static constexpr int C1 = imax(4, 1 << ((ceil_log2(C0) + 1) / 2));
  static constexpr int C2 = imax(4, C1 / 2);
  static constexpr int C3 = 1, C4 = 1;
  static constexpr int K1 = C2, K2 = 2, K3 = 1, K4 = 1;
  static constexpr bool kHasA1 = (K1 != C1);
  static constexpr int S = C0 + 3 * C1 + 5 * C2 + (L >= 3 ? 7 * C3 : 0) + (L >= 4 ? 9 * C4 : 0);
  static constexpr int NS = S + 2;               // node state: [S0, S1, Y]
  // offsets inside the node state (after the two normaliser sums)
  static constexpr int Y0 = 2;
  static constexpr int Y1 = Y0 + C0;              // [3][C1]
  static constexpr int Y2 = Y1 + 3 * C1;          // [5][C2]
  static constexpr int Y3 = Y2 + 5 * C2;          // [7]
  static constexpr int Y4 = Y3 + (L >= 3 ? 7 : 0); // [9]
  // lane mapping of the edge kernels: LPE lanes per edge, lane k owns the
  // channels c = k + LPE*j, j < CPL, so channel c < C1 sits in slot j = 0
  static constexpr int LPE = C1;
  static constexpr int CPL = C0 / LPE;
  static constexpr int EPW = kWave / LPE;
  static constexpr int PW = 2 + R;                // pair cache entries per channel
  // descriptor layout, Eq. (descriptor)
  // (triples in lexicographic order, Eq. (triples): (1,1,2) (1,2,3) (1,3,4)
  // (2,2,2) (2,2,4) (2,3,3) (2,4,4) (3,3,4) (4,4,4))
  static constexpr int nG1 = C1 * (C1 + 1) / 2, nG2 = C2 * (C2 + 1) / 2, nG3 = (L >= 3 ? 1 : 0);
  static constexpr int nG4 = (L >= 4 ? 1 : 0);
  static constexpr int n112 = K1 * (K1 + 1) / 2 * K2;
  static constexpr int n123 = (L >= 3 ? K1 * K2 * K3 : 0);
  static constexpr int n134 = (L >= 4 ? K1 : 0);
  static constexpr int n222 = K2 * (K2 + 1) * (K2 + 2) / 6;
  static constexpr int n224 = (L >= 4 ? K2 * (K2 + 1) / 2 : 0);
  static constexpr int n233 = (L >= 3 ? K2 : 0);
  static constexpr int n244 = (L >= 4 ? K2 : 0);
  static constexpr int n334 = (L >= 4 ? 1 : 0), n444 = (L >= 4 ? 1 : 0);
  static constexpr int nPi = K2 * K1;
  static constexpr int oX0 = 0, oX = C0, oM0 = 2 * C0, oM1 = 2 * C0 + 1;
  static constexpr int oG1 = 2 * C0 + 2, oG2 = oG1 + nG1, oG3 = oG2 + nG2, oG4 = oG3 + nG3;
  static constexpr int o112 = oG4 + nG4, o123 = o112 + n112, o134 = o123 + n123;
  static constexpr int o222 = o134 + n134, o224 = o222 + n222, o233 = o224 + n224;
  static constexpr int o244 = o233 + n233, o334 = o244 + n244, o444 = o334 + n334;
  static constexpr int oPi = o444 + n444;
  static constexpr int DOUT = oPi + nPi;
  static constexpr int DSTR = (DOUT + 15) / 16 * 16;   // row stride of descriptor arrays
  static_assert(C0 % LPE == 0, "channel split");
  static_assert(R == 0 || R == 4, "the edge kernels handle 0 or 4 radial modes");
  static_assert(L >= 2 && L <= 4, "degrees 2 to 4");
  static_assert(kWave % LPE == 0, "edge groups");
};

// The compiled profiles: the five DPA4C variants of Supplementary Table S3,
// each with its MLP width.
using NanoProfile = Profile<8, 2, 0>;      // MLP width 96
using MiniProfile = Profile<32, 2, 0>;     // 192
using NeoProfile = Profile<64, 2, 0>;      // 256
using AirProfile = Profile<64, 3, 4>;      // 256
using PlusProfile = Profile<128, 3, 4>;    // 384
// the Plus widths with harmonics up to degree four (nine coupling triples)
using PlusL4Profile = Profile<128, 4, 4>;  // 384
static_assert(NanoProfile::DOUT == 70 && NanoProfile::S == 40, "Table S2 (8, 2)");
static_assert(MiniProfile::DOUT == 144 && MiniProfile::S == 76, "Table S2 (32, 2)");
static_assert(NeoProfile::DOUT == 208 && NeoProfile::S == 108, "Table S2 (64, 2)");
static_assert(AirProfile::DOUT == 219 && AirProfile::S == 115, "Table S2 (64, 3)");
static_assert(PlusProfile::DOUT == 541 && PlusProfile::S == 223, "Table S2 (128, 3)");
static_assert(PlusL4Profile::DOUT == 557 && PlusL4Profile::S == 232, "Table S2 (128, 4)");

// Calls fn(P{}, std::integral_constant<int, F>{}) for the compiled profile
// matching (C0, L, R) and MLP width F and returns its result; returns
// kNoProfile when none matches.
constexpr int kNoProfile = -1000;
template <class Fn>
int with_profile(int C0, int L, int R, int F, Fn&& fn) {
  if (C0 == 8 && L == 2 && R == 0 && F == 96) return fn(NanoProfile{}, std::integral_constant<int, 96>{});
  if (C0 == 32 && L == 2 && R == 0 && F == 192) return fn(MiniProfile{}, std::integral_constant<int, 192>{});
  if (C0 == 64 && L == 2 && R == 0 && F == 256) return fn(NeoProfile{}, std::integral_constant<int, 256>{});
  if (C0 == 64 && L == 3 && R == 4 && F == 256) return fn(AirProfile{}, std::integral_constant<int, 256>{});
  if (C0 == 128 && L == 3 && R == 4 && F == 384) return fn(PlusProfile{}, std::integral_constant<int, 384>{});
  if (C0 == 128 && L == 4 && R == 4 && F == 384) return fn(PlusL4Profile{}, std::integral_constant<int, 384>{});
  return kNoProfile;
}

// ---------------------------------------------------------------------------
// Device-side view of a model, passed to kernels by value.
// ---------------------------------------------------------------------------
constexpr int kMaxTypeRows = 128;        // type-table rows (species + padding) a model may have
constexpr int kMaxFoldTypes = 5;         // species for which pair-folded tables are built
constexpr size_t kMaxFoldBytes = size_t(256) << 20;  // and their largest total size
constexpr int kC123 = 3 * 5 * 7;          // dense (1,2,3) coupling, [m1][m2][m3]
constexpr int kC233 = 5 * 7 * 7;          // dense (2,3,3) coupling
constexpr int kCouplings = kC123 + kC233;
// degree four adds (1,3,4), (2,2,4), (2,4,4), (3,3,4), (4,4,4), dense, in
// that order after the degree-three pair
constexpr int kC134 = 3 * 7 * 9, kC224 = 5 * 5 * 9, kC244 = 5 * 9 * 9, kC334 = 7 * 7 * 9,
              kC444 = 9 * 9 * 9;
constexpr int kO134 = kCouplings, kO224 = kO134 + kC134, kO244 = kO224 + kC224,
              kO334 = kO244 + kC244, kO444 = kO334 + kC334;
constexpr int kCouplings4 = kO444 + kC444;
// couplings stored for a maximum degree L
constexpr int couplings_for(int L) { return L >= 4 ? kCouplings4 : (L >= 3 ? kCouplings : 0); }

struct ModelDev {
  // radial table: g rows [n_rows][CPL][LPE][6], q rows [n_rows][R][6]
  const float* gtab;
  const float* qtab;
  int n_rows;
  float inv_delta;
  float r_c;
  float inv_rc;             // 1 / r_c
  int n_types1;             // T + 1
  const float* pair;        // [(T+1)^2][CPL][LPE][PW]
  const float* type_embed;  // [T+1][C0]
  const float* W1;          // [C1][C1] alignment, degree 1 (I + W applied in-kernel)
  const float* W2;          // [C2][C2]
  const float* A1;          // [C1][K1] or null (identity)
  const float* A2;          // [C2][K2]
  const float* mu;          // [D_out]
  const float* inv_sigma;   // [D_out]
  const float* cpl;         // [kCouplings]: C123 then C233 (symmetric in m2, m3), or null
  const float* E_ref;       // [T+1]
  // pair-folded tables (fold.hip), used when fold_n > 0:
  // [fold_n^2 pairs][n_rows] rows of kFoldWords C0 words in the order of
  // load_fold_row, pair (fa, fb) at fa * fold_n + fb; c_inv = the inverse
  // scales of the float16 c2, c3
  const float* ftab;
  int fold_n;
  float c_inv[4];
};

// Words per channel of a folded table: c0 and c1 as float32, then (c2, c3)
// as a scaled float16 pair: one 12-byte load.
constexpr int kFoldWords = 3;

// ---------------------------------------------------------------------------
// Error handling
// ---------------------------------------------------------------------------
void set_error(const std::string& msg);

// a failed HIP call returns DPA4C_ERR_OOM when the device (or pinned host)
// memory is exhausted, DPA4C_ERR_HIP otherwise
#define DPA4C_HIP_TRY(expr)                                                      \
  do {                                                                           \
    hipError_t _e = (expr);                                                      \
    if (_e != hipSuccess) {                                                      \
      ::dpa4c::set_error(std::string(#expr) + ": " + hipGetErrorString(_e));     \
      return _e == hipErrorOutOfMemory ? DPA4C_ERR_OOM : DPA4C_ERR_HIP;          \
    }                                                                            \
  } while (0)

// returns the (negative) code of a failed library call
#define DPA4C_TRY(expr)        \
  do {                         \
    const int _r = (expr);     \
    if (_r) return _r;         \
  } while (0)

// packed image shift: ((nx+128) << 16) | ((ny+128) << 8) | (nz+128)
__host__ __device__ inline int32_t pack_shift(int nx, int ny, int nz) {
  return ((nx + 128) << 16) | ((ny + 128) << 8) | (nz + 128);
}
__host__ __device__ inline int unpack_x(int32_t s) { return ((s >> 16) & 0xFF) - 128; }
__host__ __device__ inline int unpack_y(int32_t s) { return ((s >> 8) & 0xFF) - 128; }
__host__ __device__ inline int unpack_z(int32_t s) { return (s & 0xFF) - 128; }
// shift of the reverse edge: n -> -n
__host__ __device__ inline int32_t negate_shift(int32_t s) {
  return pack_shift(-unpack_x(s), -unpack_y(s), -unpack_z(s));
}

}  // namespace dpa4c
