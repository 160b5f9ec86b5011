/*
 * dpa4c.h -- C ABI of the MI355X (gfx950) energy-and-force path of the DPA4C
 * machine-learning potential (arXiv 2608.19041).
 *
 * The library evaluates, for N atoms with positions r_i, species a_i and a
 * periodic cell (orthorhombic or triclinic), the neighbour graph of Methods Eq.
 * (neighbor-set), the single message-passing layer of Eqs. (edge-geometry)
 * .. (moments), the invariant readout and MLP of Eqs. (alignment) ..
 * (fitting), and the forces of Eq. (forces), F_k = -dE/dr_k.  The compressed
 * execution of Methods "Compressed inference" is used: the radial maps g(rho)
 * and q(rho) come from a quintic Hermite table (Supplementary Note "Quintic
 * Hermite interpolation of the radial table"), the ordered-pair modulation
 * from a per-pair cache; everything else is analytic.
 *
 * Units: Angstrom, eV, fs, atomic mass units (u).
 *
 * Pointers marked "device" are HIP device pointers on the model's device;
 * pointers marked "host" are ordinary host memory.  The caller owns every
 * array passed in; the library owns only what hangs off a model handle
 * (weights, tables, caches, a grow-only workspace) and a small per-device
 * workspace of build_neighbors.  All device work is enqueued on ``stream``
 * (a hipStream_t; NULL = the default stream) and runs asynchronously unless
 * stated otherwise; inputs must stay valid until the stream reaches that
 * point.
 *
 * Every function returns 0 on success or a negative DPA4C_ERR_* code; on
 * failure dpa4c_last_error() describes the problem.  Nothing is written to
 * caller outputs on failure, except where a function says so.
 *
 * Calls that share a model handle must not overlap (the handle's workspace
 * is shared); different handles may be used concurrently.
 */
#ifndef DPA4C_H
#define DPA4C_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DPA4C_OK 0
#define DPA4C_ERR_INVALID_ARG (-1) /* bad pointer, size or value */
#define DPA4C_ERR_UNSUPPORTED (-2) /* open axes of a non-diagonal cell, profile not built, row too long */
#define DPA4C_ERR_CAPACITY (-3)    /* neighbour capacity too small; *n_pairs holds the need */
#define DPA4C_ERR_HIP (-4)         /* a HIP runtime call failed */
#define DPA4C_ERR_NONFINITE (-5)   /* a non-finite position was found */
#define DPA4C_ERR_SKIN (-6)        /* an atom moved more than half the skin, rebuild disabled */
#define DPA4C_ERR_OOM (-7)         /* device memory exhausted (hipErrorOutOfMemory); nothing was
                                      computed, the model stays usable with a smaller input */

typedef struct dpa4c_model dpa4c_model;

/*
 * Weight blob (little endian).  A 64-byte header
 *     char magic[8] = "DPA4CW01"; int32 version = 1;
 *     int32 C0, L, R, n_rbf, F (MLP width), n_layers (Lambda), n_types (T);
 *     float64 r_c, delta (radial-table spacing, Angstrom); zero padding,
 * followed by float32 row-major arrays in this order (widths per Methods
 * Eqs. (degree-channels), (probe-ranks), (dim-out); H = 8 ceil(C0/3),
 * Hp = 8 ceil(2 C0/3), K1 = C2, K2 = 2):
 *     type_embed [T+1][C0]      Eq. (init-features); row T is the zero padding type
 *     omega      [n_rbf]        Eq. (bessel-basis)
 *     W_in       [n_rbf][2H]    Eq. (radial-map); gate = first H columns
 *     W_out      [H][C0]
 *     W_mode     [H][R]         Eq. (radial-modes)
 *     Wp_in      [2 C0][2 Hp]   Eq. (pairfilm); gate = first Hp columns
 *     Wp_out     [Hp][C0 (2+R)] output split [s, t, w], w channel-major (C0, R)
 *     W_align1   [C1][C1], W_align2 [C2][C2]   Eq. (alignment)
 *     A1         [C1][K1]       Eq. (probes); only when K1 != C1
 *     A2         [C2][K2]
 *     Theta1 [D_out][F], b1 [F], then Theta_t [F][F], b_t [F] for t = 2..Lambda
 *     w_head [F], b_head [1]    Eq. (fitting)
 *     E_ref  [T+1]              Eq. (atomic-energy)
 *     mu [D_out], sigma [D_out] Eq. (calibration)
 * Supported (C0, L, R, F): the five variants of Supplementary Table S3,
 * (8,2,0,96) (32,2,0,192) (64,2,0,256) (64,3,4,256) (128,3,4,384), and the
 * Plus widths with harmonics up to degree four, (128,4,4,384), each with
 * n_layers = 3 for the per-atom kernel; others fail with UNSUPPORTED, as
 * does n_types > 127 (the type table, padding row included, holds at most
 * 128 rows).
 *
 * Creates a model on ``device``: uploads the weights, tabulates [g, q] on
 * knots rho_s = s*delta (values and first two derivatives evaluated in
 * float64, quintic coefficients stored float32), evaluates the ordered-pair
 * cache for all (T+1)^2 pairs, and builds the Gaunt coupling tensors of
 * Eq. (gaunt).  Synchronous.  *out receives the handle.
 */
int dpa4c_model_create(const void* blob, size_t nbytes, int device, dpa4c_model** out);

/* Frees the handle and everything it owns (synchronises its device). */
void dpa4c_model_destroy(dpa4c_model* model);

/*
 * Integer widths of a model, written to ``info`` (host, 13 int64):
 * C0, L, R, S (Eq. (moment-width)), D_out (Eq. (dim-out)), F, n_layers,
 * n_types, table rows, C1, C2, K1, and the words per channel of its folded
 * radial tables (3: c0, c1 in float32 and c2, c3 in scaled float16, the
 * quintic's c4, c5 being below float32 resolution for this model; 0: the
 * model runs on the separable float32 tables only).
 */
int dpa4c_model_info(const dpa4c_model* model, int64_t* info);

/*
 * Neighbour list of Eq. (neighbor-set) at radius r_list (typically r_c plus
 * a skin), for a periodic cell (orthorhombic or triclinic) or an open or
 * partly open system.  Along an open axis no periodic image is a neighbour.
 *
 * Membership uses the exact fixed-point predicate
 *     |Q(r_j) + sum_b n_b Q(h_b) - Q(r_i)|^2 < Q(r_list)^2,  Q(x) = rint(x * 2^20)
 * (Q of every component of every lattice vector h_b)
 * in 64-bit integers, so the list is a deterministic function of the float64
 * positions.  Periodic images are distinct neighbours, only (j = i, n = 0)
 * is excluded, both orientations are stored and there is no capacity per
 * atom.  Rows are in canonical order: ascending (j, n_x, n_y, n_z).
 * Positions need not lie inside the cell.
 *
 * pos       device float64 [N][3]
 * cell      host float64 [9], rows are the lattice vectors h_0, h_1, h_2
 *           (any non-singular matrix, entries below 1e6 A; a diagonal cell
 *           must have a positive diagonal), or NULL for an open system
 * pbc       host int [3] (ignored when cell is NULL): pbc[a] = 0 opens axis
 *           a, which needs a diagonal cell (its length on open axes is not
 *           used).  Internally an open axis is given the length
 *           extent + 2 r_list + 1 A, read from the positions (one more
 *           synchronisation), so no image can be within r_list
 * row_ptr   device int64 [N+1] out: CSR row offsets
 * nbr_j     device int32 [cap] out: neighbour index j
 * nbr_shift device int32 [cap] out: image n packed as
 *           ((n_x+128) << 16) | ((n_y+128) << 8) | (n_z+128), |n_a| <= 127
 * n_pairs   host out: number of edges; always set when the count succeeded.
 * If the edge count exceeds cap, returns DPA4C_ERR_CAPACITY with *n_pairs
 * set and row_ptr written, but nbr_j / nbr_shift untouched; call again with
 * cap >= *n_pairs.  A non-finite position gives DPA4C_ERR_NONFINITE; an
 * image index beyond +-127 gives DPA4C_ERR_UNSUPPORTED.  Rows have no length
 * limit (rows beyond 512 entries are ordered through a device scratch of
 * 8 bytes per entry, allocated when the count finds one).  Synchronises
 * ``stream`` twice (to read the count and the error flags).
 */
int build_neighbors(const double* pos, int64_t N, const double cell[9], const int pbc[3],
                    double r_list, int64_t* row_ptr, int32_t* nbr_j, int32_t* nbr_shift,
                    int64_t cap, int64_t* n_pairs, void* stream);

/*
 * Energy and forces for one configuration (Eqs. (energy-decomposition),
 * (atomic-energy), (forces)).
 *
 * The neighbour list passed in is a skin list from build_neighbors (same
 * cell and pbc) at any radius r_list >= r_c built for positions from which
 * no atom has moved by more than (r_list - r_c)/2 (integer norm); the
 * library keeps the edges with
 * the r_c predicate itself, in canonical order.  r_c must equal the model's.
 * n_pairs is the number of edges of that list (row_ptr[N], as returned by
 * build_neighbors); it sizes the library's edge workspace.
 *
 * pos      device float64 [N][3];  species device int32 [N], 0 <= a < T
 * e_atom   device float64 [N] out: E_i
 * forces   device float64 [N][3] out
 * e_total  device float64 [1] out: sum of E_i (fixed-order two-pass sum)
 * All reductions run in a fixed order without floating-point atomics, so
 * repeated calls give bit-identical results.  Synchronises ``stream`` once,
 * to read the species present and the list's size back.
 *
 * The list is checked on the device before anything is written: if
 * row_ptr[N] exceeds n_pairs, or some entry (i -> j, n) has no reverse
 * (j -> i, -n) (a list that is not symmetric), the call returns
 * DPA4C_ERR_INVALID_ARG.
 */
int compute_energy_forces(const dpa4c_model* model, const double* pos, const int32_t* species,
                          int64_t N, const double cell[9], const int pbc[3], double r_c,
                          const int64_t* row_ptr, const int32_t* nbr_j, const int32_t* nbr_shift,
                          int64_t n_pairs, double* e_atom, double* forces, double* e_total,
                          void* stream);

/*
 * compute_energy_forces plus the virial of Eq. (forces),
 *     Xi = -sum_i sum_{j in N_i} dE/dr_ij (x) r_ij      (eV),
 * from the same per-edge gradients: r_ij is the float64 difference stored in
 * float32, products and sums are float64, in a fixed order.  The stress is
 * -Xi / V (Methods, benchmark metrics).
 *
 * virial       device float64 [9] out (required): Xi[a][b], row-major
 * atom_virial  device float64 [N][9] out, or NULL: the per-centre terms
 *              W_i = -sum_{j in N_i} dE/dr_ij (x) r_ij, which sum to Xi
 * Other arguments, errors and determinism as compute_energy_forces.
 */
int compute_energy_forces_virial(const dpa4c_model* model, const double* pos,
                                 const int32_t* species, int64_t N, const double cell[9],
                                 const int pbc[3], double r_c, const int64_t* row_ptr,
                                 const int32_t* nbr_j, const int32_t* nbr_shift, int64_t n_pairs,
                                 double* e_atom, double* forces, double* e_total, double* virial,
                                 double* atom_virial, void* stream);

/*
 * compute_energy_forces without any device allocation, for callers that
 * cannot allocate while they run: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc.  Same arguments, outputs,
 * determinism and errors as compute_energy_forces; the library calls no
 * hipMalloc, hipFree or allocating routine and records no memset.
 *
 * The per-call buffers live in a fixed 64 MiB device array (one per device,
 * held until the process ends) instead of the model's workspace.  They take
 * 28 bytes per list entry (n_pairs), 8 (S+2) + 8 bytes per atom and about
 * 1 KB more (each array rounded up to 256 bytes): about 12,000 atoms of a
 * dense metal at the full width with a 1 A skin.  A larger input returns
 * DPA4C_ERR_INVALID_ARG before any device work.  Every call on a device
 * shares that device's array, so calls that overlap on one device (other
 * streams, other threads, other models) race; calls on one stream do not.
 *
 * The pair-folded radial tables are built only inside the allocation a
 * previous call on the model left: with a species set whose tables do not
 * fit it, this call reads the separable tables (the same model, results
 * equal to float32 rounding).  One compute_energy_forces call with the same
 * species beforehand gives this entry point the folded tables.  The model's
 * own workspace, and so the list that verlet_step carries between calls, is
 * untouched.  Synchronises ``stream`` once (the species present).
 */
int compute_energy_forces_noalloc(const dpa4c_model* model, const double* pos,
                                  const int32_t* species, int64_t N, const double cell[9],
                                  const int pbc[3], double r_c, const int64_t* row_ptr,
                                  const int32_t* nbr_j, const int32_t* nbr_shift, int64_t n_pairs,
                                  double* e_atom, double* forces, double* e_total, void* stream);

/*
 * ``nsteps`` velocity-Verlet NVE steps (Supplementary Note on the MD
 * protocol: full neighbour list with a skin, checked every step):
 *     v += dt/2 F/m;  r += dt v;  [rebuild];  F = F(r);  v += dt/2 F/m.
 * The library keeps its own skin list (radius r_c + skin) in the model
 * workspace.  It is rebuilt at the first step of a call, every
 * ``rebuild_every`` steps when that is > 0, and at every step where some
 * atom has moved by more than skin/2 since the last build (fixed-point
 * check on the device).  With rebuild_every == 0, a periodic cell and the
 * list of the model's previous call still in place (same N, cell and
 * radius, and no compute_energy_forces call since), the first step is
 * checked like any other instead of rebuilt: results do not depend on which
 * valid list is used, so a run split over several calls equals one call.  The steps between builds run in batches that the
 * host checks after the fact: a batch that contains such a step is rolled
 * back to its saved start (positions, velocities, forces), the steps before
 * the violation are replayed and the violating step rebuilds, so the
 * trajectory is the one a per-step check gives, bit for bit.  With
 * rebuild_every < 0 no rebuild happens after the first step and a violation
 * returns DPA4C_ERR_SKIN (pos, vel, forces then hold the state at the end of
 * a batch that contains the violating step).
 *
 * pos, vel         device float64 [N][3], in/out (A, A/fs)
 * species          device int32 [N]
 * mass_by_species  host float64 [T+1] (u)
 * forces           device float64 [N][3]: in = forces at the input
 *                  positions (from compute_energy_forces or a previous call);
 *                  out = forces at the final positions
 * e_pot, e_kin     device float64 [nsteps] out: potential and kinetic energy
 *                  after each step (eV)
 * n_rebuilds       host int64 out (may be NULL): rebuilds done in this call
 * Synchronises ``stream`` once per batch and at every rebuild (to size the
 * skin list: its capacity grows to the pair count plus 1/8 and 16 per atom
 * whenever a build needs more).  The workspace holds 36 bytes per slot of
 * that capacity, 72 N bytes for the batch start state and the node state;
 * an allocation that would leave less than 512 MiB of device memory free
 * returns DPA4C_ERR_OOM.
 */
int verlet_step(const dpa4c_model* model, double* pos, double* vel, const int32_t* species,
                const double* mass_by_species, int64_t N, const double cell[9], const int pbc[3],
                double r_c, double skin, double dt_fs, int nsteps, int rebuild_every,
                double* e_pot, double* e_kin, double* forces, int64_t* n_rebuilds, void* stream);

/*
 * ``nsteps`` NVT steps with a Nose-Hoover chain thermostat (the paper's
 * whole-step benchmark propagates NVT at 300 K): the chain of Martyna, Klein
 * and Tuckerman (J. Chem. Phys. 97, 2635, 1992), propagated over half steps
 * by the Trotter factorisation of Martyna, Tuckerman, Tobias and Klein (Mol.
 * Phys. 87, 1117, 1996).  Per step:
 *     chain dt/2;  v += dt/2 F/m;  r += dt v;  [rebuild];  F = F(r);
 *     v += dt/2 F/m;  chain dt/2,
 * where a chain half step scales all velocities by exp(-dt/2 v_xi1).  Chain
 * masses Q_1 = N_f kT tau^2 and Q_k = kT tau^2 (tau = t_damp_fs), with
 * N_f = 3N - 3.  The virial of Eq. (forces) is assembled at every step.
 * Neighbour list, rebuilds, batches and replay as verlet_step; the chain
 * state is saved with the batch start state.  Between two steps the closing
 * half step scales the velocities, and the opening one starts from the
 * kinetic energy of the scaled velocities, as it must at the start of a
 * call, so a run split over several calls equals one call, bit for bit.
 *
 * temperature      target T (K), > 0
 * t_damp_fs        damping time tau (fs), > 0
 * chain_length     M, 1..8
 * chain            device float64 [2M], in/out: xi_1..xi_M then v_xi1..v_xiM
 *                  (zeros for a fresh thermostat)
 * e_pot, e_kin     device float64 [nsteps] out: potential and kinetic energy
 *                  after each step (eV)
 * e_thermo         device float64 [nsteps] out: thermostat energy after each
 *                  step, sum Q_k v_k^2/2 + N_f kT xi_1 + kT sum_{k>1} xi_k;
 *                  e_pot + e_kin + e_thermo is the conserved quantity
 * virial           device float64 [nsteps][9] out, or NULL: Xi at each step
 * Other arguments, errors and synchronisation as verlet_step; N >= 2.
 */
int nvt_step(const dpa4c_model* model, double* pos, double* vel, const int32_t* species,
             const double* mass_by_species, int64_t N, const double cell[9], const int pbc[3],
             double r_c, double skin, double dt_fs, int nsteps, int rebuild_every,
             double temperature, double t_damp_fs, int chain_length, double* chain,
             double* e_pot, double* e_kin, double* e_thermo, double* virial, double* forces,
             int64_t* n_rebuilds, void* stream);

/*
 * Intermediate quantities of the last compute_energy_forces (or the last
 * step of verlet_step) on this model, copied into caller device buffers,
 * for stage-by-stage checks.  Any pointer may be NULL.
 *   node_state  float32 [N][S+2]: [sum chi^2, sum chi^4, unnormalised
 *               features Y (degree -> m -> channel)]   Eq. (payload)
 *   descriptor  float32 [N][D_out]: calibrated D       Eq. (calibration)
 *   edge_count  int32 [N]: edges within r_c per centre
 * The stages are recomputed from the inputs of that call (positions,
 * species and skin list), which must still hold the same values.
 * Synchronous on ``stream``.
 */
int dpa4c_debug_stages(const dpa4c_model* model, int64_t N, float* node_state,
                       float* descriptor, int32_t* edge_count, void* stream);

/*
 * Per-stage timing.  For every stage s whose bit (1 << s) is set in
 * ``stage_mask`` (0: none, -1: all), the library records HIP events around
 * the kernels of that stage on the caller's stream and accumulates their
 * durations.  The events cost a few microseconds per stage and launch, so
 * timing only the stage of interest keeps a timed run close to an untimed
 * one.  dpa4c_get_timings writes up to ``n`` stage times (milliseconds,
 * summed over calls since the last read) to ``ms``, launch counts to
 * ``count`` (either may be NULL) and returns the number of stages;
 * dpa4c_stage_name gives their names.  Reading synchronises the device.
 */
int dpa4c_set_timing(dpa4c_model* model, int64_t stage_mask);
int dpa4c_get_timings(dpa4c_model* model, double* ms, int64_t* count, int n);
const char* dpa4c_stage_name(int stage);

/*
 * C = A B for row-major float32 A [M][K], B [K][N], C [M][N] (device), with
 * K a multiple of 16 and N a multiple of 4: the fp32 matrix-core GEMM of the
 * MLP stage, exported so that tests can check it against a reference.
 */
int dpa4c_debug_gemm(const float* A, const float* B, float* C, int M, int N, int K,
                     void* stream);

/* Thread-local description of the last error (library-owned string). */
const char* dpa4c_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DPA4C_H */
