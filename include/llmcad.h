/*
 * llmcad.h — C ABI of the MI355X (gfx950) token-tree verification library.
 *
 * The library computes the target model's side of LLMCad's
 * generate-then-verify decoding (arXiv 2309.04255):
 *
 *   §3.2 "Token tree verification and rectification": one non-autoregressive
 *   pass of the target model over every node of a draft token tree, where a
 *   node only sees the accepted prefix and its own branch (the masking table of
 *   §3.2 "Tree decoder"), followed by the greedy acceptance of the longest
 *   root path whose draft tokens equal the target's output (branch correct
 *   sequences and the depth-first verified-sequence search of §3.2).
 *
 * The model is a LLaMA-style decoder (the paper names only embedding, masked
 * self-attention, norm and linear layers, §2.1): RMSNorm, rotary positions
 * (rotate-half pairing), multi-head attention, SwiGLU feed-forward, untied LM
 * head, no biases.  Weights and the KV cache are bf16; matrix products
 * accumulate in fp32; the residual stream and logits are fp32.
 *
 * Conventions shared by every entry point
 *  - All device buffers are owned by the caller; the library never allocates,
 *    frees or synchronises.  Work is enqueued on `stream` (a hipStream_t passed
 *    as void*; NULL = the null stream) and results are valid once the caller
 *    has synchronised that stream.
 *  - Return value: LLMCAD_OK (0) or a negative status (see below).  Every
 *    argument check happens on the host before anything is enqueued; on error
 *    nothing is enqueued and no device buffer (in particular the KV cache) is
 *    touched.  Device faults surface at the caller's synchronisation.
 *  - Calls that share a workspace must not overlap (same stream serialises).
 *
 * Data layouts (row-major, bf16 = IEEE bfloat16 bit pattern)
 *  - Plain weights, W[out][in]:
 *      tok_embed [V][d], final_norm [d], lm_head [V][d]
 *      per layer: attn_norm [d], w_qkv [3d][d] (rows q, then k, then v),
 *                 w_o [d][d], ffn_norm [d],
 *                 w_gate_up [2F][d] (rows gate, then up), w_down [d][F]
 *  - Packed weights: an opaque device image of llmcad_packed_bytes() bytes
 *    written by llmcad_pack_globals / llmcad_pack_layer (MFMA-fragment order:
 *    1 KiB contiguous per 16 output columns x 32 inputs, consecutive inputs
 *    consecutive).  The globals sit
 *    first, then layer 0, 1, ...; an image packed for L layers also serves a
 *    configuration with fewer layers.
 *  - KV cache: k_cache is bf16 [L][H][capacity][Dh] and v_cache is bf16
 *    [L][H][Dh][capacity] (V transposed per head: a slot is one entry of each
 *    of the head's Dh rows, so that both operands of the attention's products
 *    load from the cache in matrix-core fragment order).  capacity must be a
 *    multiple of 64 (so that every V row starts on a 128-byte line).  Slot p
 *    holds position p of the accepted sequence for p < prefix_len.
 */
#ifndef LLMCAD_H
#define LLMCAD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define LLMCAD_OK 0
#define LLMCAD_EARG (-1)       /* NULL pointer, bad config value, bad layer index   */
#define LLMCAD_ETREE (-2)      /* n < 1 or n > max, parent[0] != -1, parent[i] not
                                  in [0, i), token outside [0, V)                    */
#define LLMCAD_ECAPACITY (-3)  /* prefix_len < 0, prefix_len + n > capacity, or
                                  capacity not a positive multiple of 64             */
#define LLMCAD_ESHAPE (-4)     /* unsupported shape (see llmcad_check_config)       */
#define LLMCAD_EHIP (-5)       /* a HIP launch or runtime call failed               */
#define LLMCAD_EWORKSPACE (-6) /* workspace or packed image smaller than required   */

/* Largest tree (number of nodes) one verification pass accepts; also the
 * largest chunk a prefill pass processes at once. */
#define LLMCAD_MAX_NODES 128

typedef struct llmcad_config {
  int32_t n_layers;  /* L                                            */
  int32_t d_model;   /* d = n_heads * head_dim, a multiple of 64     */
  int32_t n_heads;   /* H (as many K/V heads as query heads)         */
  int32_t head_dim;  /* Dh, 64 or 128                                */
  int32_t d_ffn;     /* F (SwiGLU hidden width), any value >= 1      */
  int32_t vocab;     /* V                                            */
  float rms_eps;     /* RMSNorm epsilon                              */
  float rope_theta;  /* rotary base: pair j rotates at theta^(-2j/Dh) */
  int32_t weight_bits; /* layer matrices: 16 (or 0) = bf16; 4 = group-quantised
                          4-bit codes (see llmcad_pack_layer_q4; d and d_ffn
                          multiples of 128).  Embedding, LM head and norm gains
                          are bf16 either way.                                */
} llmcad_config;

typedef struct llmcad_layer_weights {
  const void* attn_norm; /* device bf16 [d]      */
  const void* w_qkv;     /* device bf16 [3d][d]  */
  const void* w_o;       /* device bf16 [d][d]   */
  const void* ffn_norm;  /* device bf16 [d]      */
  const void* w_gate_up; /* device bf16 [2F][d]  */
  const void* w_down;    /* device bf16 [d][F]   */
} llmcad_layer_weights;

/* Checks a configuration: LLMCAD_OK, LLMCAD_EARG (non-positive sizes, bad
 * eps/theta, weight_bits not 0/16/4) or LLMCAD_ESHAPE (head_dim not 64/128,
 * d != H*Dh, d % 64 != 0; with weight_bits 4, d or d_ffn not a multiple of
 * 128). */
int llmcad_check_config(const llmcad_config* cfg);

/* Bytes of the packed weight image for cfg (0 if cfg is invalid). */
size_t llmcad_packed_bytes(const llmcad_config* cfg);

/* Re-lays the model-wide tensors (embedding, final norm, LM head) from the
 * plain layouts above into the packed image.  Source buffers may be freed
 * once the stream has passed this call. */
int llmcad_pack_globals(const llmcad_config* cfg, const void* tok_embed, const void* final_norm,
                        const void* lm_head, void* packed, size_t packed_bytes, void* stream);

/* Re-lays one layer's weights (layer in [0, L)) into the packed image
 * (bf16 configurations; LLMCAD_EARG for weight_bits 4). */
int llmcad_pack_layer(const llmcad_config* cfg, int32_t layer, const llmcad_layer_weights* src,
                      void* packed, size_t packed_bytes, void* stream);

/*
 * 4-bit weights (the paper's phone targets are 4-bit models quantised with
 * AutoGPTQ, §4.1 "Models and datasets"; GPTQ's symmetric group-wise form):
 * a matrix W[out][in] is given as codes q[out][in] in [0, 16), two per byte
 * (input 2j in the low nibble of byte j: uint8 [out][in / 2]), and bf16
 * scales s[out][in / 128]; the weight it stands for is
 *     w[o][i] = s[o][i / 128] * (q[o][i] - 8).
 * The pass multiplies the codes on the matrix cores and applies each group's
 * scales to its partial sums (in fp32): the dequantised matrix is never
 * formed, and only the codes and scales cross HBM.
 */
typedef struct llmcad_q4_matrix {
  const void* codes;  /* device uint8 [out][in / 2] */
  const void* scales; /* device bf16 [out][in / 128] */
} llmcad_q4_matrix;

typedef struct llmcad_q4_layer_weights {
  const void* attn_norm;     /* device bf16 [d]          */
  llmcad_q4_matrix w_qkv;    /* [3d][d] (rows q, k, v)    */
  llmcad_q4_matrix w_o;      /* [d][d]                    */
  const void* ffn_norm;      /* device bf16 [d]          */
  llmcad_q4_matrix w_gate_up;/* [2F][d] (rows gate, up)   */
  llmcad_q4_matrix w_down;   /* [d][F]                    */
} llmcad_q4_layer_weights;

/* Re-lays one layer's 4-bit weights (weight_bits 4 configurations only, else
 * LLMCAD_EARG) into the packed image; the globals are packed with
 * llmcad_pack_globals as for bf16 models. */
int llmcad_pack_layer_q4(const llmcad_config* cfg, int32_t layer, const llmcad_q4_layer_weights* src,
                         void* packed, size_t packed_bytes, void* stream);

/* Bytes of workspace for passes of up to max_n nodes (max_n in [1, 128]) on
 * the current device (the split of the work, and so the size, depends on its
 * compute-unit count). */
size_t llmcad_workspace_bytes(const llmcad_config* cfg, int32_t max_n);

/* Clears the workspace's synchronisation counters and its zero block.  Call
 * once after allocating a workspace (a zero-filled allocation needs no call);
 * every pass leaves the counters cleared again and never writes the zero
 * block. */
int llmcad_workspace_init(const llmcad_config* cfg, int32_t max_n, void* workspace,
                          size_t workspace_bytes, void* stream);

/*
 * One verification pass over a token tree (§3.2).
 *
 * Tree (host arrays, read before the call returns): n nodes in topological
 * order; tree_tokens[0] is the root, the last accepted token, which is not yet
 * in the KV cache; parent[0] = -1 and 0 <= parent[i] < i.  Node i sits at
 * position prefix_len + depth(i) and attends to cache slots [0, prefix_len)
 * plus its ancestors and itself.
 *
 * Effects and outputs (device buffers):
 *  - K/V of node i (every layer) are written to cache slot prefix_len + i; slots
 *    [0, prefix_len) are only read.  Calling again with the same arguments gives
 *    the same results.
 *  - logits: fp32 [n][V], row i = the target's logits after node i's branch
 *    (NULL: not stored).
 *  - path: int32 [n]; path[0] = 0 and path[1..accept_len] are the accepted
 *    draft nodes root-first; entries past accept_len are -1.
 *  - accept_len: int32 [1], number of accepted draft nodes (root excluded):
 *    the deepest node whose whole branch matches the target's greedy tokens
 *    (lowest node index among equally deep ones; lowest vocabulary index among
 *    equal logits).
 *  - next_token: int32 [1], the target's greedy token after the last accepted
 *    node (a rectification if that node has children, else a bonus token).
 * Requires n <= the max_n the workspace was sized for.
 */
int llmcad_verify_tree(const llmcad_config* cfg, const void* packed, void* k_cache, void* v_cache,
                       int32_t capacity, int32_t prefix_len, const int32_t* tree_tokens,
                       const int32_t* parent, int32_t n, float* logits, int32_t* path,
                       int32_t* accept_len, int32_t* next_token, void* workspace,
                       size_t workspace_bytes, void* stream);

/* Size of the scratch buffer behind llmcad_verify_tree_noalloc: 96 MiB of
 * device memory per device, enough for any pass whose workspace fits
 * (llmcad_workspace_bytes(cfg, n) <= this; e.g. the LLaMA-7B shape up to
 * n = 32, the LLaMA-13B shape up to n = 16). */
#define LLMCAD_SCRATCH_BYTES (96u << 20)

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): one
 * verification pass exactly as llmcad_verify_tree -- same arguments, checks,
 * kernels and outputs -- with the workspace replaced by a scratch buffer the
 * library holds itself, LLMCAD_SCRATCH_BYTES of device memory on each device
 * it runs on, from the first call on that device until the process ends.
 *
 * The call allocates and frees nothing.  It enqueues on `stream` a clear of
 * the scratch's synchronisation state (the scratch keeps the previous call's
 * contents), the pass, and, when status is not NULL, a copy of the pass's
 * device status to status (device int32 [1]: 0 = ok, 1 = a wait of the pass
 * ran out of its bounded spin and the outputs are invalid; see region 5 of
 * llmcad_workspace_region).  Every call on one device uses that device's one
 * scratch: calls that overlap on a device (different streams or threads)
 * race and must be serialised by the caller.
 *
 * Errors (checked on the host, nothing enqueued): as llmcad_verify_tree, and
 * LLMCAD_EWORKSPACE when the pass needs more workspace than the scratch holds;
 * LLMCAD_EHIP when the scratch's device address cannot be obtained.
 */
int llmcad_verify_tree_noalloc(const llmcad_config* cfg, const void* packed, void* k_cache, void* v_cache,
                               int32_t capacity, int32_t prefix_len, const int32_t* tree_tokens,
                               const int32_t* parent, int32_t n, float* logits, int32_t* path,
                               int32_t* accept_len, int32_t* next_token, int32_t* status, void* stream);

/*
 * Prefill: runs tokens[0..n_tokens) (host array) as positions
 * [start_pos, start_pos + n_tokens) against cache slots [0, start_pos),
 * writing their K/V to slots [start_pos, start_pos + n_tokens).  Processed in
 * chains of at most max_n tokens (the workspace's size).  last_logits (device
 * fp32 [V], NULL = not needed) receives the logits after the last token.
 */
int llmcad_prefill(const llmcad_config* cfg, const void* packed, void* k_cache, void* v_cache,
                   int32_t capacity, const int32_t* tokens, int32_t n_tokens, int32_t start_pos,
                   float* last_logits, void* workspace, size_t workspace_bytes, void* stream);

/*
 * One step of the tree decoder (§3.2 "Token tree generation", tree decoder):
 * the forward of nodes [first, n) of a token tree whose nodes [0, first)
 * were computed by earlier calls on the same cache, prefix_len and tree.
 *
 * The tree arrays are as for llmcad_verify_tree (host, all n nodes; node i
 * at position prefix_len + depth(i)).  Each computed node attends to the
 * prefix and to its ancestors and itself -- the masking table of the tree
 * decoder -- reading the earlier nodes' keys/values from their cache slots
 * prefix_len + i, and its own K/V are written to slot prefix_len + i.
 * logits: device fp32 [n - first][V], row r = the model's logits after node
 * first + r (NULL: not stored).  With first = 0 this is the forward part of
 * a verification pass; no argmax, path or next token is produced.  A draft
 * model grows its tree with calls of one new node each (first = n - 1).
 * Asynchronous on `stream`; allocates nothing.
 *
 * Errors (checked on the host, nothing enqueued): as llmcad_verify_tree, and
 * LLMCAD_ETREE unless 0 <= first < n; the workspace must hold a pass over
 * n - first rows (llmcad_workspace_bytes with max_n >= n - first).
 */
int llmcad_extend_tree(const llmcad_config* cfg, const void* packed, void* k_cache, void* v_cache,
                       int32_t capacity, int32_t prefix_len, const int32_t* tree_tokens, const int32_t* parent,
                       int32_t n, int32_t first, float* logits, void* workspace, size_t workspace_bytes,
                       void* stream);

/*
 * A computed row's next-token distribution, summarised on the device for
 * draft-tree growth (§3.1: the most likely token always extends the branch,
 * and any other token whose probability exceeds the branch threshold starts a
 * new branch; §3.2 Eq. 1: the branch pacer weighs candidates by their
 * cumulative confidence).  Probabilities are the softmax of the row's fp32
 * logits, exp(logit - max_logit) / sum_exp, in fp32.
 */
#define LLMCAD_CAND_MAX 64
typedef struct {
  int32_t count;     /* entries in tok/prob (1 .. LLMCAD_CAND_MAX); -1: more tokens than
                        LLMCAD_CAND_MAX - 1 exceed the threshold (read the logits row instead) */
  int32_t argmax;    /* the most likely token (lowest index among equal maxima) */
  float max_logit;   /* the row's largest logit */
  float sum_exp;     /* sum over the vocabulary of exp(logit - max_logit), fp32 */
  int32_t tok[LLMCAD_CAND_MAX];  /* tok[0] = argmax, then every other token with probability >
                                    threshold, by probability, higher first (ties: lower token first) */
  float prob[LLMCAD_CAND_MAX];   /* their probabilities */
} llmcad_candidates;

/*
 * A tree-decoder step (as llmcad_extend_tree) that also summarises each
 * computed row's distribution: cand (device, [n - first] records, caller
 * owned) receives, for row r (node first + r), the argmax, the softmax
 * normaliser and every token whose probability exceeds `threshold`, so a
 * draft driver reads back a few hundred bytes per fed node instead of the
 * whole logits row.  logits (device fp32 [n - first][V]) is required: the
 * summary is taken from the stored row.  The workgroup that completes the
 * LM head's argmax builds the summaries at the end of the pass, in the same
 * launch.  Asynchronous on `stream`; allocates nothing.
 *
 * Errors (checked on the host, nothing enqueued): as llmcad_extend_tree;
 * LLMCAD_EARG if logits or cand is NULL or threshold is not in (0, 1).
 */
int llmcad_extend_tree_candidates(const llmcad_config* cfg, const void* packed, void* k_cache, void* v_cache,
                                  int32_t capacity, int32_t prefix_len, const int32_t* tree_tokens,
                                  const int32_t* parent, int32_t n, int32_t first, float threshold, float* logits,
                                  llmcad_candidates* cand, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Rollback to the verified sequence after a verification pass (§3.2 "Token
 * tree verification and rectification": the tree is rolled back to the
 * verified sequence, which becomes the new input; §3.1: generation then
 * continues from the target's token after it).
 *
 * path and accept_len are device buffers holding llmcad_verify_tree's outputs
 * for a tree of n nodes verified at prefix_len (they are read on the stream,
 * after that pass).  For every layer and head, the keys and values of cache
 * slot prefix_len + path[k] move to slot prefix_len + k, k = 1..accept_len
 * (path[0] = 0, the root, is in place).  The cache then holds the accepted
 * sequence -- the prefix, the root and the accepted draft tokens, each at the
 * position it was verified at -- in slots [0, prefix_len + accept_len + 1):
 * the next pass uses prefix_len' = prefix_len + accept_len + 1 with the
 * returned next token as its root.  Slots past that are left as they are.
 * Asynchronous on `stream`; allocates nothing.
 *
 * Errors (checked on the host, nothing enqueued): LLMCAD_EARG for a NULL
 * pointer, LLMCAD_ETREE unless 1 <= n <= 128, LLMCAD_ECAPACITY unless
 * 0 <= prefix_len and prefix_len + n <= capacity.  Device-side values
 * outside what a pass over n nodes writes (accept_len not in [0, n), an entry
 * path[k] not in [k, n)) move nothing for the affected rows.
 */
int llmcad_commit_path(const llmcad_config* cfg, void* k_cache, void* v_cache, int32_t capacity,
                       int32_t prefix_len, const int32_t* path, const int32_t* accept_len, int32_t n,
                       void* stream);

/* Static text for a status code. */
const char* llmcad_status_string(int status);

/* Byte offset and size of a named intermediate buffer inside a workspace
 * sized for max_n (for diagnostics).  "Fragment order" stores a bf16 [Mp][K]
 * matrix as 1 KiB blocks, block (k-step s, row block b) at (s Mp/16 + b) KiB,
 * its 16-byte lane l holding row 16 b + l % 16, columns 32 s + 8 (l / 16) ..
 * + 7.  0 final residual stream fp32 [Mp][d], 1 layer 0's queries after the
 * rotary embedding bf16 [Mp][d], 2 layer 0's attention output bf16 [Mp][d]
 * in fragment order, 3 layer 0's SwiGLU product bf16 [Mp][Fp] in fragment
 * order, 4 per-node greedy token int32 [Mp],
 * 5 pass status int32 (0 = ok; 1 = a grid wait of the single-launch pass ran
 * out of its bounded spin: the pass's outputs are invalid, and the workspace
 * must be cleared with llmcad_workspace_init before the next pass; 3 = the
 * kernel did not find its parameter block where it reads it, and did
 * nothing),
 * 6 phase timestamps int64 [G][4 + 5L][8], G the pass's workgroups (written when the environment
 * variable LLMCAD_TRACE is 1), 7 every residual stream version fp32
 * [2L+1][Mp][d], 8 their per-16-column sums of squares fp32 [2L+1][d/16][Mp],
 * 9 every layer's queries bf16 [L][Mp][d], 10 attention outputs bf16
 * [L] x [Mp][d] in fragment order, 11 SwiGLU products bf16 [L] x [Mp][Fp]
 * in fragment order, 12 every residual stream version times the gain of the
 * RMSNorm that reads it, bf16 [2L+1] x [Mp][d] in fragment order (the input
 * of the QKV, gate/up and LM-head products), 13 the line of zeros that the
 * kernels read in place of absent inputs (cleared by llmcad_workspace_init);
 * Mp = max_n rounded up to 16, 32, 64 or 128, Fp = F rounded up to 32.  Offsets describe a
 * pass over max_n nodes (call with max_n = that pass's n); those of regions 5
 * and 13, which hold state from one pass to the next, depend on neither the
 * node count nor the pass's grid. */
int llmcad_workspace_region(const llmcad_config* cfg, int32_t max_n, int32_t which, size_t* offset,
                            size_t* bytes);

/* Kernel classes for llmcad_timing_enable.  A verification or prefill pass
 * is one persistent launch. */
#define LLMCAD_KERNEL_PASS 0

/* Diagnostics (measurement only, process-wide, not thread-safe): after
 * llmcad_timing_enable(c, m), the next m launches of kernel class c made by
 * passes are each bracketed by a pair of HIP events on the pass's stream.
 * kernel_class < 0 disables and releases the events.  llmcad_timing_read
 * waits for the recorded events, returns the summed milliseconds and the
 * number of bracketed launches, and makes the slots available again. */
int llmcad_timing_enable(int32_t kernel_class, int32_t max_launches);
int llmcad_timing_read(int32_t kernel_class, double* total_ms, int32_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* LLMCAD_H */
