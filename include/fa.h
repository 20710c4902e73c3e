/*
 * fa.h -- C ABI of libfa: encrypted nearest-neighbour scoring under RNS-CKKS
 * on one AMD Instinct MI355X (gfx950).
 *
 * What it computes (paper: "Billion-Scale Nearest-Neighbor Search under Fully
 * Homomorphic Encryption on a Single GPU, Balancing Leakage and Cost"):
 *   - the server-side scorer: one slot-packed encrypted query against blocks
 *     of up to N/2 plaintext candidate rows, each block stored as d diagonals
 *     pre-rotated by their giant step (Section 2, "Measured prototype vs.
 *     deployment" and "Reproducing this"; Section 3.1, "Detail");
 *   - the encrypted rank reduction Enc(W^T q) by the diagonal method with one
 *     final fold (Section 3.1, "How" and "Detail");
 *   - the rotate-and-sum fold and the row-packed variant;
 *   - scoring at a dropped level, batches of queries per pass over the
 *     blocks, and blocks of encrypted candidates (ct x ct);
 *   - the membership path: rescaling, ciphertext products, a Chebyshev series
 *     of the threshold and the sign iteration (Section 3.1, "Membership
 *     search");
 *   - client-side helpers for tests and benchmarks: key generation, secret-key
 *     encryption, decryption, encoding and decoding (Section 2, "Setting" and
 *     "The round trip").
 *
 * Scheme and conventions (shared with the documentation of every call):
 *   N = 2^log_n ring degree, S = N/2 slots, L ciphertext primes, K special
 *   primes, all in (2^49, 2^50) and congruent to 1 mod 2N: by default the L+K
 *   largest such primes below 2^50, in descending order.  Hybrid key switching
 *   uses alpha = K primes per digit and dnum = ceil(L/K) digits.  Slot j is
 *   the evaluation at zeta^(5^j mod 2N), zeta = exp(i*pi/N); rotating by r
 *   rolls the slots left by r (automorphism X -> X^(5^r)).  The scoring calls
 *   do not rescale: the scale of a product is the product of the scales.  The
 *   membership calls (fa_rescale onwards) rescale after every ciphertext
 *   product and track the scale as a double.
 *
 * Buffers.  Ciphertexts, plaintexts and workspaces are caller-owned DEVICE
 * memory (for example torch tensors), 8-byte words, 256-byte aligned.  Every
 * scoring-path call takes its ciphertexts and plaintexts as fa_buf
 * descriptors: the device pointer and its capacity, plus what the buffer
 * holds -- polynomials per object (2 ciphertext, 1 plaintext, 3 a product
 * before relinearisation), the number of objects stored back to back, the
 * number of primes per polynomial (its level) and the scale exponent.  One
 * object occupies n_polys * limbs * N words: a ciphertext [c0 | c1], each
 * [limbs][N]; a plaintext [limbs][N].  Calls check the descriptors of their
 * inputs on the host before any launch and return FA_E_SHAPE when a buffer is
 * at another level than the context, holds the wrong kind of object, holds too
 * few objects for the call, is smaller than its contents, or carries a scale
 * the call cannot combine (see each call).  An output descriptor must bring
 * `dev` and `bytes`; the call fills in its n_polys, count, limbs and
 * log_scale.  The word format and coefficient order inside device buffers are
 * private to the library (NTT form); fa_export_coeffs() returns the canonical
 * form: coefficient order, residues in [0, q_i) as uint64.  Host arrays are
 * marked "host".  The context owns its tables and rotation keys (device
 * memory it allocates at fa_ctx_create / fa_keygen and frees at
 * fa_ctx_destroy); the scoring calls allocate nothing.
 *
 * Streams.  Calls that take `stream` (a hipStream_t) only enqueue work on it
 * and return; the caller synchronises.  Calls without `stream` are
 * synchronous.  Some calls also use auxiliary streams of the context (default
 * priority), forked from and joined back to `stream` with events, so their
 * work is ordered on `stream` as a whole.  A context is used by one host
 * thread at a time: its auxiliary streams and events are shared.
 *
 * Errors.  Every call returns FA_OK (0) or a negative FA_E_* code; all
 * argument checks happen on the host before any launch, so a failed call has
 * enqueued nothing.  fa_last_error() returns a message for the calling
 * thread's most recent failure.  No C++ exception crosses this interface.
 */
#ifndef FA_H_
#define FA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  FA_OK = 0,
  FA_E_INVAL = -1, /* bad argument value (null pointer, out-of-range size)   */
  FA_E_SHAPE = -2, /* sizes, levels, kinds or scales inconsistent with the
                      context or with each other                             */
  FA_E_NOKEY = -3, /* a rotation key the operation needs was never generated */
  FA_E_NOMEM = -4, /* workspace too small, or a setup-time allocation failed */
  FA_E_HIP = -5    /* HIP runtime / launch error                             */
};

enum { FA_LAYOUT_ROW = 0, FA_LAYOUT_DIAG = 1, FA_LAYOUT_DIAG_ENC = 2 };
enum {
  FA_OP_SCORE = 0,
  FA_OP_PROJECT = 1,
  FA_OP_ROTATE_SUM = 2,
  FA_OP_ROTATE = 3,
  FA_OP_PREPARE = 4,
  FA_OP_SCORE_PREPARED = 5,
  FA_OP_SCORE_ENC = 6,
  FA_OP_PROJECT_ENC = 7
};

typedef struct fa_ctx fa_ctx;

typedef struct {
  uint32_t log_n;         /* 10..16 */
  uint32_t L;             /* ciphertext primes, 1..16 */
  uint32_t K;             /* special primes, 1..4 (= primes per key-switch digit); ceil(L/K) <= 8 */
  uint32_t log_scale;     /* default scale 2^log_scale of fa_encode_db_block / fa_encode_projection */
  const uint64_t* primes; /* host [L+K]: q_0..q_{L-1}, then p_0..p_{K-1}, distinct primes in
                             (2^49, 2^50), each 1 mod 2N; or NULL for the default choice */
} fa_params;

/* A caller-owned device buffer and its contents (see "Buffers" above). */
typedef struct {
  void* dev;         /* device memory, 256-byte aligned                        */
  size_t bytes;      /* its capacity in bytes                                  */
  uint32_t n_polys;  /* polynomials per object: 2 ciphertext, 1 plaintext      */
  uint32_t count;    /* objects stored back to back                            */
  uint32_t limbs;    /* primes per polynomial: the level                       */
  int32_t log_scale; /* the objects are at scale 2^log_scale                   */
} fa_buf;

/* ---- context ------------------------------------------------------------ */

/* Create a context on the current HIP device for the scheme parameters of
 * Section 2 "Security parameters" (ring degree, RNS primes, scale): selects
 * or checks the primes, builds twiddle and basis-conversion tables on the
 * device.  Returns FA_E_INVAL for parameters outside the ranges of fa_params
 * (including more than 8 key-switch digits, and explicit primes that are not
 * distinct primes in (2^49, 2^50) congruent to 1 mod 2N) before touching the
 * device, FA_E_NOMEM / FA_E_HIP on device failure.  *out is set only on
 * success. */
int fa_ctx_create(const fa_params* params, fa_ctx** out);
void fa_ctx_destroy(fa_ctx* ctx);

/* A lower-level context over the first L_low ciphertext primes of `parent`
 * and the same special primes (same N, K, scale).  Its secret and every
 * rotation key are the parent's restricted to those primes: a key digit's
 * gadget P*Qhat_i*[Qhat_i^-1]_{Q_i} is P on the digit's own primes and 0 on
 * the others at every level, so the restriction is the lower-level key.  The
 * database can then live at this shallow level (the paper stores it at the
 * level its ranked product needs, Section 2 "Measured prototype vs.
 * deployment").  Keys generated later on either context are not shared. */
int fa_ctx_create_level(const fa_ctx* parent, uint32_t L_low, fa_ctx** out);
/* Level drop of `ct` (ciphertexts of `parent`, at parent->L primes) to the
 * level of `child` (fa_ctx_create_level): keeps the first child L limbs of c0
 * and c1 of every ciphertext, scale unchanged.  Exact while the message plus
 * noise stays below half the product of the kept primes.  FA_E_SHAPE if
 * `child` is not a lower level of `parent` or ct is not at the parent's
 * level. */
int fa_drop_level(const fa_ctx* parent, const fa_ctx* child, const fa_buf* ct, fa_buf* out, void* stream);

/* The L+K primes (host out[L+K]): q_0..q_{L-1}, then p_0..p_{K-1}. */
int fa_ctx_primes(const fa_ctx* ctx, uint64_t* out);
size_t fa_ct_bytes(const fa_ctx* ctx);  /* one ciphertext: 2*L*N*8 */
size_t fa_pt_bytes(const fa_ctx* ctx);  /* one plaintext:    L*N*8 */
size_t fa_key_bytes(const fa_ctx* ctx); /* device bytes per rotation key */
const char* fa_last_error(void);

/* ---- keys and client-side operations (tests, benchmark set-up) ---------- */

/* Rotation keys (the keys a rotation of the packed vector needs, Section 2
 * "What CKKS gives us"; the server keeps them resident, Section 3.4
 * "Warm-query kernel path") for left rotations by steps[0..n_steps-1]
 * (1 <= step < S), switching from the automorphed secret sigma_{5^r}(s) back
 * to s, with all randomness supplied by the caller (host arrays):
 *   s  [N]                        ternary secret, entries in {-1, 0, 1}
 *   a  [n_steps][dnum][L+K][N]    uniform residues, a[..][t][..] < prime t
 *   e  [n_steps][dnum][N]         small noise integers
 * Key digit i of step r: b_i = -a_i*s + e_i + (P*Qhat_i*[Qhat_i^-1]_{Q_i})*sigma(s)
 * over every prime of Q u P.  Keys already present for a step are replaced.
 * Synchronous; allocates the keys' device memory.  Errors: FA_E_INVAL (null
 * array, a step out of range, a non-ternary secret), FA_E_NOMEM, FA_E_HIP. */
int fa_keygen(fa_ctx* ctx, const int64_t* s, const int32_t* steps, int n_steps, const uint64_t* a,
              const int64_t* e);
/* 1 if a key for left rotation by `step` exists, else 0. */
int fa_has_key(const fa_ctx* ctx, int step);

/* Relinearisation key for ct x ct products (the encrypted-database scoring of
 * Section 2, "Measured prototype vs. deployment", where the stored rows are
 * ciphertexts): the rotation-key form with s^2 in place of sigma(s),
 *   b_i = -a_i*s + e_i + (P*Qhat_i*[Qhat_i^-1]_{Q_i}) * s^2  over Q u P,
 * with the same host inputs as one step of fa_keygen (a [dnum][L+K][N],
 * e [dnum][N]).  Replaces an existing relinearisation key; synchronous. */
int fa_keygen_relin(fa_ctx* ctx, const int64_t* s, const uint64_t* a, const int64_t* e);
/* 1 if the relinearisation key exists, else 0. */
int fa_has_relin_key(const fa_ctx* ctx);

/* Secret-key encryption of the query by its owner (Section 2 "The round
 * trip", step 1; the single-key setting of "Setting"): host inputs
 *   m [N] integer plaintext coefficients (|m| < 2^62) at scale 2^log_scale,
 *   a [L][N] uniform residues, e [N] noise (|e| <= 1024); s is the secret
 *   given to fa_keygen (or set by fa_set_secret).
 * Writes one ciphertext c1 = a, c0 = -a*s + e + m into ct (device; its
 * descriptor gets n_polys 2, count 1, limbs L, log_scale).  Synchronous on
 * the stream.  Errors: FA_E_INVAL (null pointer, a coefficient out of range),
 * FA_E_SHAPE (ct->bytes below one ciphertext), FA_E_NOMEM / FA_E_HIP. */
int fa_set_secret(fa_ctx* ctx, const int64_t* s);
int fa_encrypt(fa_ctx* ctx, const int64_t* m, int32_t log_scale, const uint64_t* a, const int64_t* e, fa_buf* ct,
               void* stream);
/* Encrypts the pts->count device plaintexts of `pts` (as written by
 * fa_encode_db_block / fa_encode_db_block_int) into cts (device, that many
 * ciphertexts, same scale): ct_j = (-a_j*s + e_j + pt_j, a_j) with host
 * a [count][L][N] residues and e [count][N] noise (|e| <= 1024).  This is how
 * a data owner enrolls an encrypted block (FA_LAYOUT_DIAG_ENC; Section 2
 * "Measured prototype vs. deployment": a deployment stores the database as
 * ciphertexts).  Synchronous on the stream. */
int fa_encrypt_pts(fa_ctx* ctx, const fa_buf* pts, const uint64_t* a, const int64_t* e, fa_buf* cts, void* stream);
/* The client's decryption of a score ciphertext (Section 2 "The round trip",
 * steps 3, 5 and 7): m' = c0 + c1*s of the first ciphertext of ct,
 * coefficient form, host out [L][N] residues in [0, q_i).  Synchronous with
 * respect to `stream`.  FA_E_SHAPE unless ct holds a ciphertext at the
 * context's level. */
int fa_decrypt(fa_ctx* ctx, const fa_buf* ct, uint64_t* out, void* stream);
/* Canonical form of every polynomial of a device buffer: host out
 * [count][n_polys][L][N], coefficient order, residues in [0, q_i) -- the
 * representation in which ciphertexts are compared word for word with an
 * independent implementation of the scheme (Section 2 "What CKKS gives us").
 * Synchronous on the stream.  FA_E_SHAPE unless buf is at the context's
 * level. */
int fa_export_coeffs(fa_ctx* ctx, const fa_buf* buf, uint64_t* out, void* stream);
/* The inverse of fa_export_coeffs: buf->count objects of buf->n_polys
 * polynomials in canonical form (host [count][n_polys][L][N], limb t of
 * every polynomial below prime t) into buf (device) in the library's
 * private form; buf->limbs must be L and buf->log_scale is kept.  Enrolled
 * blocks can so be saved and loaded again without re-encoding them (the
 * paper keeps its encrypted database on disk and reloads it warm, Section 2
 * "Measured prototype vs. deployment").  Allocates a staging buffer;
 * synchronous on the stream.  Errors: FA_E_INVAL (null pointer, a residue
 * not below its prime), FA_E_SHAPE (limbs, n_polys or capacity), FA_E_NOMEM,
 * FA_E_HIP. */
int fa_import_coeffs(fa_ctx* ctx, const uint64_t* coeffs, fa_buf* buf, void* stream);
/* Encode a real slot vector (host, n_slots <= S values, rest zero) to integer
 * coefficients m_k = rint(2^log_scale * (2/N) * sum_j v_j cos(pi k 5^j / N))
 * (round half to even, float64): host out [N] (the client's packing of its
 * query into slots, Section 2 "What CKKS gives us"). */
int fa_encode(const fa_ctx* ctx, const double* slots, int n_slots, int log_scale, int64_t* out);
/* Decode decrypted residues (host [L][N], e.g. from fa_decrypt) at scale
 * 2^log_scale into n_slots real slot values (host): the client's reading of
 * its scores (Section 2 "The round trip").  The centred CRT uses the first
 * primes whose product exceeds 2^(log_scale + 22), which is exact for slot
 * values of magnitude below 2^12 (scores are cosines).  Runs on the calling
 * thread only and touches no device state: a client may decode several
 * blocks at once from threads of its own. */
int fa_decode(const fa_ctx* ctx, const uint64_t* res, int log_scale, double* out, int n_slots);

/* ---- server: enrollment ------------------------------------------------- */

/* Encode a block of candidate rows (host float32 [n_rows][dim], dim <= d,
 * zero-padded to d) into device plaintexts at scale 2^(ctx log_scale):
 *   FA_LAYOUT_DIAG (Section 2 "Measured prototype vs. deployment": a block of
 *     n/2 vectors stored as its diagonals; Section 3.1 "Detail": each
 *     diagonal pre-rotated in plaintext by its giant-step amount): n_rows <= S;
 *     d diagonals diag_j[i] = X[i][(i+j) mod d], diagonal gB+b pre-rotated
 *     right by gB, stored g-major: pts[g*B+b]; d % baby_step == 0, d | S.
 *     Writes d plaintexts.
 *   FA_LAYOUT_ROW: rows packed S/d per plaintext, slot t*d+u = X[w*S/d+t][u];
 *     writes ceil(n_rows / (S/d)) plaintexts (baby_step ignored).
 * pts->bytes must hold that many plaintexts; its descriptor is filled in
 * (n_polys 1, count, limbs L, log_scale).  Errors: FA_E_SHAPE (d not a power
 * of two <= S, dim outside [1, d], no rows or more than S rows in a diagonal
 * block, pts too small), FA_E_INVAL (null pointer, unknown layout, baby step
 * not dividing d). */
int fa_encode_db_block(fa_ctx* ctx, const float* rows, int n_rows, int dim, int d, int layout, int baby_step,
                       fa_buf* pts, void* stream);
/* Plaintexts of a projection W (host float32 [d_in][r], row-major) for
 * fa_project_ct (Section 3.1 "How", "Detail"): the r hybrid diagonals
 * e_j[s] = W[(s+j) mod d_in][s mod r] over all S slots, diagonal gB+b
 * pre-rotated right by gB, stored g-major (pts[g*B+b]), at scale
 * 2^(ctx log_scale).  d_in and r powers of two, r | d_in, d_in | S,
 * baby_step | r.  Writes r plaintexts. */
int fa_encode_projection(fa_ctx* ctx, const float* W, int d_in, int r, int baby_step, fa_buf* pts, void* stream);
/* Plaintexts from integer coefficients (host [n_pts][N], |c| < 2^62, the
 * caller's encoding at scale 2^log_scale): the enrollment of the same
 * diagonal or row layouts from coefficients computed elsewhere (for example
 * by an independent encoder).  Writes n_pts plaintexts. */
int fa_encode_db_block_int(fa_ctx* ctx, const int64_t* coeffs, int n_pts, int32_t log_scale, fa_buf* pts,
                           void* stream);

/* ---- server: scoring ---------------------------------------------------- */

/* Device workspace needed by an operation (bytes).  op = FA_OP_SCORE with
 * layout FA_LAYOUT_DIAG (FA_OP_SCORE_ENC with FA_LAYOUT_DIAG_ENC): n_blocks,
 * d, baby_step as passed to fa_score_block;
 * FA_OP_PROJECT (FA_OP_PROJECT_ENC for fa_project_ct_enc): n_blocks = 1,
 * d = r; FA_OP_ROTATE_SUM / FA_OP_ROTATE: n_blocks
 * = number of ciphertexts. */
size_t fa_workspace_bytes(const fa_ctx* ctx, int op, int n_blocks, int d, int baby_step);

/* The stateless scorer of Section 2 "Reproducing this": per request it takes
 * the encrypted query and a list of group ids, gathers those groups' rows --
 * here blocks resident in HBM -- and returns their encrypted scores.
 *   q: one ciphertext (slot s = query[s mod d]) at the context's level;
 *   blocks[0..n_resident-1]: the resident blocks of this level;
 *   block_ids[0..n_blocks-1]: the blocks to score, each in [0, n_resident),
 *     repeats allowed; NULL scores blocks 0..n_blocks-1;
 *   out: n_blocks ciphertexts, out[j] the scores of block block_ids[j], at
 *     scale 2^(q log_scale + block log_scale).
 * Layouts:
 *   FA_LAYOUT_DIAG (Section 3.1 diagonal method, baby step B = baby_step,
 *   G = d/B giant steps): each block holds d pre-rotated plaintexts from
 *   fa_encode_db_block; slot i of out[j] is <X_i, q>.  Sequence:
 *   qrot_b = Rotate(q, b) (b < B, one shared decomposition);
 *   acc_g = sum_b pt[g*B+b] * qrot_b; out = acc_0 + sum_{g>=1} Rotate(acc_g, gB)
 *   with the key-switch products of all g >= 1 summed over Q u P before one
 *   division by P per block.  Needs keys for steps 1..B-1 and g*B, 1 <= g < G.
 *   FA_LAYOUT_DIAG_ENC: as FA_LAYOUT_DIAG with every block holding d
 *   ciphertexts (fa_encrypt_pts of a diagonal block): acc_g is the
 *   three-component tensor sum over b, relinearised once per (block, g)
 *   (lazy relinearisation), before the same giant steps.  Needs the
 *   relinearisation key as well.
 *   FA_LAYOUT_ROW: each block holds row-packed plaintexts, of which the first
 *   is used; out[j] = q * pt (no rotation; follow with
 *   fa_rotate_sum(first_shift=1, n_steps=log2 d)).
 * ws: device workspace of ws_bytes >= fa_workspace_bytes(...).
 * Errors: FA_E_SHAPE if n_blocks < 1 (checked first: an empty request is a
 * shape error, whatever the pointers), if d is not a power of two <= N/2, if
 * q is not one ciphertext at the context's level, if a scored block is at
 * another level, holds the wrong kind or fewer than d objects, if the scored
 * blocks are not all at one scale, if the product scale exceeds
 * 2^(log2 Q - 8) (the scores would wrap modulo Q), or if out cannot hold
 * n_blocks ciphertexts; FA_E_INVAL for a null pointer, an unknown layout, a
 * block id outside [0, n_resident) or a baby step not dividing d;
 * FA_E_NOKEY / FA_E_NOMEM for a missing key or a short workspace. */
int fa_score_block(fa_ctx* ctx, const fa_buf* q, const fa_buf* blocks, int n_resident, const int32_t* block_ids,
                   int n_blocks, int d, int layout, int baby_step, fa_buf* out, void* ws, size_t ws_bytes,
                   void* stream);

/* The same diagonal-layout scoring split in two, so that one query's baby
 * rotations serve several levels or batches (the paper projects the query
 * once and reuses it across batches, Section 3.4):
 *   fa_prepare_query writes Rotate(q, b), b = 1..baby_step-1, into prep
 *     (device, fa_prepared_bytes(ctx, baby_step) bytes; its descriptor gets
 *     n_polys 2, count baby_step-1, the query's level and scale);
 *   fa_score_prepared then scores q against blocks exactly as fa_score_block
 *     with FA_LAYOUT_DIAG does (bit-identical output); FA_E_SHAPE if prep
 *     does not hold baby_step-1 rotations at q's level and scale.
 * Workspace: FA_OP_PREPARE (baby_step) and FA_OP_SCORE_PREPARED (n_blocks,
 * d, baby_step). */
size_t fa_prepared_bytes(const fa_ctx* ctx, int baby_step);
int fa_prepare_query(fa_ctx* ctx, const fa_buf* q, int baby_step, fa_buf* prep, void* ws, size_t ws_bytes,
                     void* stream);
int fa_score_prepared(fa_ctx* ctx, const fa_buf* q, const fa_buf* prep, const fa_buf* blocks, int n_resident,
                      const int32_t* block_ids, int n_blocks, int d, int baby_step, fa_buf* out, void* ws,
                      size_t ws_bytes, void* stream);

/* Several queries prepared together (the cross-query batching of "Conclusion
 * and Future Work" applied to the baby rotations): preps[j] receives exactly
 * what fa_prepare_query(qs[j], baby_step) writes, for j < n_q.  The key
 * switches of one baby step are issued for the queries of a group together
 * (groups of at most 16 queries; from four queries on a launch group holds
 * 64 rotations), so a rotation key read from HBM for one query is found in
 * the caches by the others.  qs[j] device ciphertexts,
 * preps[j] device, fa_prepared_bytes(ctx, baby_step) bytes each; workspace
 * fa_prepare_batch_workspace_bytes(n_q, baby_step) bytes (it grows with the
 * group size: every query's extended digits).  Errors: FA_E_INVAL (null
 * pointer, baby_step out of range), FA_E_SHAPE (n_q < 1, a query not one
 * ciphertext at the context's level, a prepared buffer too small),
 * FA_E_NOKEY (a baby-step key is missing), FA_E_NOMEM (workspace too
 * small). */
size_t fa_prepare_batch_workspace_bytes(const fa_ctx* ctx, int n_q, int baby_step);
int fa_prepare_batch(fa_ctx* ctx, const fa_buf* qs, int n_q, int baby_step, fa_buf* preps, void* ws,
                     size_t ws_bytes, void* stream);

/* Cross-query batching against resident blocks ("Conclusion and Future
 * Work": score a batch of queries per loaded region so that the load is paid
 * once per batch): n_q queries, each prepared with fa_prepare_query (qs[j]
 * the query ciphertext, preps[j] its baby rotations), scored against the
 * same blocks (blocks / n_resident / block_ids as in fa_score_block).  Each
 * pass over the plaintexts serves up to four queries, so the plaintext stream
 * is read once per four queries instead of once per query.  outs[j] (device,
 * n_blocks ciphertexts) is bit-identical to fa_score_prepared(qs[j],
 * preps[j], ...).  The giant steps of all n_q queries then run together, over
 * n_q * n_blocks blocks in chunks of up to 16.  Workspace:
 * fa_batch_workspace_bytes(n_q, n_blocks, d, baby_step) bytes (the
 * accumulators of all n_q queries plus the giant-step scratch of one chunk).
 * Errors as fa_score_prepared; FA_E_SHAPE if n_q < 1. */
size_t fa_batch_workspace_bytes(const fa_ctx* ctx, int n_q, int n_blocks, int d, int baby_step);
int fa_score_batch(fa_ctx* ctx, const fa_buf* qs, const fa_buf* preps, int n_q, const fa_buf* blocks,
                   int n_resident, const int32_t* block_ids, int n_blocks, int d, int baby_step, fa_buf* outs,
                   void* ws, size_t ws_bytes, void* stream);

/* Encrypted projection q_R = W^T q (Section 3.1 "How"): q holds one
 * d_in-periodic query ciphertext, w_pts the r plaintexts of W's hybrid
 * diagonals e_j[s] = W[(s+j) mod d_in][s mod r] (j < r), encoded as a
 * FA_LAYOUT_DIAG block (pre-rotated, g-major, baby step B; Section 3.1
 * "Detail").  Runs the same baby-step/giant-step product, then one final
 * fold: z += Rotate(z, r*2^k) for k < log2(d_in/r).  Output slot
 * s = (W^T q)[s mod r], at scale 2^(q log_scale + w log_scale).  Needs keys
 * 1..B-1, g*B, and r*2^k.  Errors: FA_E_SHAPE (d_in, r not powers of two
 * with r <= d_in <= N/2; q or w_pts at another level, of the wrong kind, w_pts
 * holding fewer than r plaintexts; the product scale above 2^(log2 Q - 8);
 * q_r too small), FA_E_INVAL (null pointer, baby step not dividing r),
 * FA_E_NOKEY, FA_E_NOMEM. */
int fa_project_ct(fa_ctx* ctx, const fa_buf* q, const fa_buf* w_pts, int d_in, int r, int baby_step, fa_buf* q_r,
                  void* ws, size_t ws_bytes, void* stream);

/* The projection with W itself encrypted (Section 3.1 "How": the server holds
 * the projection's diagonals as ciphertexts).  w_cts holds r ciphertexts
 * (fa_encrypt_pts of the plaintexts fa_project_ct takes); each giant step's
 * three-component tensor sum is relinearised once, as for FA_LAYOUT_DIAG_ENC
 * blocks, before the same giant steps and fold.  Output slot
 * s = (W^T q)[s mod r] at the product of the two scales.  Needs the keys
 * fa_project_ct needs and the relinearisation key (FA_E_NOKEY otherwise).
 * Workspace: fa_workspace_bytes(FA_OP_PROJECT_ENC, 1, r, baby_step).  Other
 * errors as fa_project_ct. */
int fa_project_ct_enc(fa_ctx* ctx, const fa_buf* q, const fa_buf* w_cts, int d_in, int r, int baby_step,
                      fa_buf* q_r, void* ws, size_t ws_bytes, void* stream);

/* The rotate-and-sum fold (Section 3.1 "Detail": one final fold after the
 * diagonal product; the row-packed scoring sums a row's slots the same way):
 * in place, for each of the cts->count ciphertexts of cts,
 * ct <- ct + Rotate(ct, first_shift * 2^k) for k = 0..n_steps-1.  Errors:
 * FA_E_SHAPE (cts not ciphertexts at the context's level), FA_E_INVAL (null
 * pointer, a shift out of [1, N/2)), FA_E_NOKEY, FA_E_NOMEM. */
int fa_rotate_sum(fa_ctx* ctx, fa_buf* cts, int first_shift, int n_steps, void* ws, size_t ws_bytes, void* stream);

/* out = Rotate(ct, step): one full key switch of the first ciphertext of ct
 * (Section 2 "What CKKS gives us": rotating the packed vector).  out must not
 * overlap ct (FA_E_INVAL): the key-switch finish reads ct through the
 * automorphism while it writes out. */
int fa_rotate(fa_ctx* ctx, const fa_buf* ct, int step, fa_buf* out, void* ws, size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The same
 * rotation as fa_rotate, with its key-switch scratch (the decomposed and
 * extended digits, the special-prime sums, the conversions) in a fixed device
 * array of the library instead of a caller workspace: FA_STATIC_SCRATCH_BYTES
 * per GPU, reserved on each GPU the library runs on until the process ends.
 * The call allocates nothing.  FA_E_NOMEM if the context's rotation needs more
 * scratch than that (fa_workspace_bytes(ctx, FA_OP_ROTATE, 1, 0, 1) >
 * FA_STATIC_SCRATCH_BYTES; N=2^16 with 12+3 primes needs 63 MiB); FA_E_HIP if
 * the array could not be located on this GPU when the context was created.
 * Every call on one GPU uses that GPU's one array and leaves its contents
 * behind (nothing in it has to start at zero): calls that overlap on one GPU
 * (other streams, other host threads, other contexts) race.  Other errors as
 * fa_rotate. */
#define FA_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
int fa_rotate_static(fa_ctx* ctx, const fa_buf* ct, int step, fa_buf* out, void* stream);

/* ---- the membership (threshold) path ------------------------------------
 * Section 3.1 ("Membership search"): the server returns an encrypted yes/no
 * for score >= tau |q_R| by approximating tau |q_R| = sqrt(tau^2 |q_R|^2)
 * with a low-degree Chebyshev polynomial (direct evaluator) and then the
 * sign of score - tau |q_R| after pre-scaling into [-1, 1].  These calls run
 * on a chain of contexts, levels[0] with L primes and each next one the
 * previous minus its last ciphertext prime (fa_ctx_create_level), every one
 * holding the relinearisation key.  A ciphertext's level is its number of
 * primes and its scale is a double (after rescaling it is no power of two),
 * both passed explicitly, so these calls take plain device pointers instead
 * of fa_buf descriptors.  Products are relinearised and rescaled by the last
 * prime of their level (scale sa*sb/q); constants are integers. */

/* Rescale n_polys polynomials of ct ([n_polys][L][N] at hi) by hi's last
 * prime: out ([n_polys][L-1][N], lo's layout) = round(ct / q_last), the
 * remainder centred in (-q_last/2, q_last/2].  lo must be hi minus that prime.
 * ws: n_polys * L * N words. */
int fa_rescale(const fa_ctx* hi, const fa_ctx* lo, const void* ct, int n_polys, void* out, void* ws,
               size_t ws_bytes, void* stream);
/* out = Relin(x (x) y) at one level (no rescale); needs the relinearisation
 * key.  ws: fa_workspace_bytes is not used; pass fa_chain_workspace_bytes(ctx, 1). */
int fa_mul_ct(fa_ctx* ctx, const void* x, const void* y, void* out, void* ws, size_t ws_bytes, void* stream);
/* out = x + y (subtract = 0) or x - y; out = k * x; out = x + k (the constant
 * k on every slot: k / scale) -- k an integer (for fa_ct_add_const an
 * integer-valued double, any magnitude below 2^1000, as constants at a
 * product's scale exceed 64 bits); out may alias x. */
int fa_ct_add(fa_ctx* ctx, const void* x, const void* y, void* out, int subtract, void* stream);
int fa_ct_mul_const(fa_ctx* ctx, const void* x, int64_t k, void* out, void* stream);
int fa_ct_add_const(fa_ctx* ctx, const void* x, double k, void* out, void* stream);
/* Workspace (bytes) of fa_cheb_eval of this degree and of fa_sign_iter
 * (degree 3) on a chain whose first context is top. */
size_t fa_chain_workspace_bytes(const fa_ctx* top, int degree);
/* sum_{k<=degree} coeffs[k] T_k(u), u at level L_u and scale s_u with slots in
 * [-1, 1]: T_{a+b} = 2 T_a T_b - T_{a-b} (a = b = k/2 with T_0 = 1 for even k,
 * a = b + 1 with T_1 for odd k), T_2..T_degree in order; every T_k is then
 * dropped to the lowest level, multiplied by round(c_k q) for that level's
 * last prime q, summed with round(c_0 s_u q) and rescaled.  Writes the result
 * to out (a ciphertext at *L_out primes, scale *s_out). */
int fa_cheb_eval(fa_ctx* const* levels, int n_levels, const void* u, int L_u, double s_u, const double* coeffs,
                 int degree, void* out, int* L_out, double* s_out, void* ws, size_t ws_bytes, void* stream);
/* iters steps towards sign(x), x = V/m in [-1, 1] (m >= 1 an integer): with
 * f(x) = (3x - x^3)/2, V <- V (3 m^2 - V^2) and m <- 2 m^3 each step (two
 * levels per step, integer constants only).  out holds the last V (level
 * *L_out, scale *s_out); its value divided by *m_out approximates f^iters(x). */
int fa_sign_iter(fa_ctx* const* levels, int n_levels, const void* v, int L_v, double s_v, int64_t m, int iters,
                 void* out, int* L_out, double* s_out, int64_t* m_out, void* ws, size_t ws_bytes, void* stream);

/* Chebyshev interpolation coefficients (coeffs[0..degree]) of
 * g(u) = tau * sqrt(y(u)), y(u) = (y_lo + y_hi)/2 + u (y_hi - y_lo)/2, on
 * u in [-1, 1], at the degree + 1 Chebyshev points of the first kind: the
 * low-degree square-root approximation of the threshold tau |q_R| (Section
 * 3.1 "Membership search").  Host only.  FA_E_INVAL unless 0 < y_lo < y_hi
 * and 1 <= degree <= 64. */
int fa_cheb_fit_sqrt(double tau, double y_lo, double y_hi, int degree, double* coeffs);

/* Membership scan of one projected query against resident candidate blocks
 * (Section 3.1 "Membership search": the server decides under encryption
 * whether cos(q, x_i) >= tau, as the sign of <q_R, x_i> - tau |q_R|, with
 * |q_R| = sqrt(|q_R|^2) by a low-degree Chebyshev series, pre-scaled into
 * [-1, 1]).  levels: the chain as for fa_cheb_eval; q_r a ciphertext at level
 * L_q (scale s_q) holding the d-periodic projected query (slot s =
 * q_R[s mod d], as fa_project_ct writes it, rescaled or not); blocks[i]
 * diagonal blocks (fa_encode_db_block, FA_LAYOUT_DIAG, baby_step) encoded on
 * the chain's level-L_q context.  Steps:
 *   score_i = Rescale(diagonal product of q_r with block i)  (level L_q - 1);
 *   y = |q_R|^2 in every slot: Rescale(q_r * q_r) folded by y += Rotate(y, 2^k),
 *       2^k < d (needs level L_q - 1 keys for those steps);
 *   u = (2y - y_lo - y_hi)/(y_hi - y_lo): the factor taken into the scale,
 *       the shift an added constant;
 *   t = sum_k coeffs[k] T_k(u) (fa_cheb_eval's evaluator; coeffs from
 *       fa_cheb_fit_sqrt or any series of tau |q_R| in u), produced at the
 *       scores' scale;
 *   out_i = fa_sign_iter((score_i - t) at t's level, m, iters): with
 *       x = (score_i - t)/m in [-1, 1], out_i / *m_out approximates
 *       f^iters(x), f(x) = (3x - x^3)/2, whose sign is the decision.
 * out: n_blocks ciphertexts at a stride of 2*L_q*N words, each valid in its
 * first 2*(*L_out)*N words (level *L_out, scale *s_out).  Levels used:
 * 1 (scores) + ceil(log2 degree) + 1 (series) + 2*iters; FA_E_SHAPE if the
 * chain is too short.  ws: fa_membership_workspace_bytes(level-L_q context,
 * n_blocks, d, baby_step, degree) bytes. */
size_t fa_membership_workspace_bytes(const fa_ctx* ctx_q, int n_blocks, int d, int baby_step, int degree);
int fa_membership(fa_ctx* const* levels, int n_levels, const void* q_r, int L_q, double s_q,
                  const void* const* blocks, int n_blocks, int d, int baby_step, double y_lo, double y_hi,
                  const double* coeffs, int degree, int64_t m, int iters, void* out, int* L_out, double* s_out,
                  int64_t* m_out, void* ws, size_t ws_bytes, void* stream);

/* ---- measurement -------------------------------------------------------- */

/* Phase timing of subsequent diagonal-layout fa_score_block calls with HIP
 * events recorded on the call's stream (enable != 0 turns it on; adds no
 * synchronisation).  fa_profile_read waits for the last profiled call and
 * writes ms[0] baby rotations, ms[1] multiply-accumulate stream,
 * ms[2] giant steps, ms[3] whole call; FA_E_INVAL if nothing was profiled. */
int fa_profile(fa_ctx* ctx, int enable);
int fa_profile_read(fa_ctx* ctx, double* ms);

#ifdef __cplusplus
}
#endif
#endif /* FA_H_ */
