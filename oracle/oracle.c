/*
 * oracle.c -- TEST INFRASTRUCTURE ONLY, not part of the product.
 *
 * A plain, slow, single-threaded CPU implementation of what the trie-automaton
 * token-mask path computes, written from the paper's definitions and sharing no
 * code with the HIP library.  Only the tests, the smoke check and the bench's
 * CPU-baseline leg may load it.
 *
 * What it follows:
 *   - Section 4.1 (character-level trie): one trie over the set strings built by
 *     inserting each string character by character; one node per distinct prefix
 *     (appendix "FSM Complexity Analysis": node count = number of distinct
 *     prefixes).
 *   - Section 4.1 and appendix "Correctness", conditions (i) and (ii): token v is
 *     valid at node n iff the bytes of v, walked from n, never fall off the trie.
 *     Condition (ii) (an accept state stays reachable) holds for every trie node,
 *     so the walk surviving is the whole test.
 *   - The naive precomputation of Section 4.1 / appendix "Precomputation Cost
 *     Breakdown": check every token at every node by simulating the walk.  That
 *     is exactly what oracle_mask_rows does, one byte at a time.
 *   - Section 2, Eq. (1): the constrained distribution zeroes the probability of
 *     every token outside the valid set, i.e. its logit becomes -inf.
 *   - Section 2: the next state is the character-level transition function
 *     extended over the sampled token's bytes (oracle_advance).
 *
 * Readings where the paper is silent (each also listed in the design notes):
 *   - End of a value: instead of an EOS token, every string is followed by a
 *     terminator byte T (default '"') that is inserted as an ordinary trie edge.
 *     The node after T is final and has no children, so tokens that overshoot a
 *     completed value (e.g. '",') fall off the trie and are invalid.
 *   - A set string that contains T is rejected (error 2).
 *   - Duplicate set strings collapse (set semantics); the empty string is allowed.
 *   - Node ids: rank of the prefix in bytewise lexicographic order, a proper
 *     prefix before its extensions (= DFS preorder, children in ascending byte
 *     order), root = 0.  A forest of S sets numbers set j after sets 0..j-1.
 *   - The dead state is -1.  A node id or token id out of range is dead.  An
 *     empty token has no character decomposition (the paper's special tokens)
 *     and is never valid.
 *   - Mask rows: W = ceil(V/64) little-endian 64-bit words; token v is bit v&63
 *     of word v>>6; bits at or beyond V are 0.
 *   - Apply: in place; valid entries keep their exact bits, invalid ones become
 *     -inf (fp32 0xFF800000, bf16 0xFF80).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <stdio.h>

#define OR_OK 0
#define OR_E_INVAL 1
#define OR_E_TERMINATOR 2
#define OR_E_NOMEM 3

static char g_err[256];

const char *oracle_last_error(void) { return g_err; }

/* ---------------------------------------------------------------- build --- */

/* A pointer trie node during construction: children kept sorted by byte. */
typedef struct {
    int nchild, cap;
    uint8_t *cbyte;
    int *cnode;
} pnode;

typedef struct {
    pnode *v;
    int n, cap;
} ptrie;

static int ptrie_new_node(ptrie *t) {
    if (t->n == t->cap) {
        int nc = t->cap ? t->cap * 2 : 64;
        pnode *nv = (pnode *)realloc(t->v, (size_t)nc * sizeof(pnode));
        if (!nv) return -1;
        t->v = nv;
        t->cap = nc;
    }
    memset(&t->v[t->n], 0, sizeof(pnode));
    return t->n++;
}

/* Child of node p along byte c, or -1. */
static int ptrie_child(const ptrie *t, int p, uint8_t c) {
    const pnode *nd = &t->v[p];
    for (int i = 0; i < nd->nchild; i++)
        if (nd->cbyte[i] == c) return nd->cnode[i];
    return -1;
}

/* Child of node p along byte c, created (keeping the byte order) if absent. */
static int ptrie_child_or_add(ptrie *t, int p, uint8_t c) {
    int q = ptrie_child(t, p, c);
    if (q >= 0) return q;
    q = ptrie_new_node(t);
    if (q < 0) return -1;
    pnode *nd = &t->v[p]; /* t->v may have moved inside ptrie_new_node */
    if (nd->nchild == nd->cap) {
        int nc = nd->cap ? nd->cap * 2 : 2;
        uint8_t *nb = (uint8_t *)realloc(nd->cbyte, (size_t)nc);
        if (!nb) return -1;
        nd->cbyte = nb;
        int *nn = (int *)realloc(nd->cnode, (size_t)nc * sizeof(int));
        if (!nn) return -1;
        nd->cnode = nn;
        nd->cap = nc;
    }
    int i = nd->nchild;
    while (i > 0 && nd->cbyte[i - 1] > c) {
        nd->cbyte[i] = nd->cbyte[i - 1];
        nd->cnode[i] = nd->cnode[i - 1];
        i--;
    }
    nd->cbyte[i] = c;
    nd->cnode[i] = q;
    nd->nchild++;
    return q;
}

static void ptrie_free(ptrie *t) {
    for (int i = 0; i < t->n; i++) {
        free(t->v[i].cbyte);
        free(t->v[i].cnode);
    }
    free(t->v);
}

/* The finished trie, numbered in preorder; children of node n are
 * kid_node[kid_off[n] .. kid_off[n+1]) with bytes kid_byte[...] ascending. */
typedef struct oracle {
    int64_t N, S;
    int64_t *kid_off;
    uint8_t *kid_byte;
    int32_t *kid_node;
    int32_t *parent;
    int32_t *depth;
    uint8_t *edge;
    uint8_t *is_final;
    int32_t *roots;
    int terminator;
} oracle;

void oracle_free(oracle *o) {
    if (!o) return;
    free(o->kid_off);
    free(o->kid_byte);
    free(o->kid_node);
    free(o->parent);
    free(o->depth);
    free(o->edge);
    free(o->is_final);
    free(o->roots);
    free(o);
}

/*
 * Build the trie of one set (Section 4.1: insert every string s followed by the
 * terminator, one byte at a time; shared prefixes merge), then renumber its
 * nodes in DFS preorder with children in ascending byte order.  Returns the
 * pointer trie and the preorder permutation order[k] = pointer-trie node of
 * preorder rank k.
 */
static int build_set(const uint8_t *sb, const int64_t *so, int64_t k0, int64_t k1, int T,
                     ptrie *t, int **order_out) {
    t->v = NULL;
    t->n = t->cap = 0;
    if (ptrie_new_node(t) != 0) return OR_E_NOMEM;
    for (int64_t k = k0; k < k1; k++) {
        int64_t a = so[k], b = so[k + 1];
        for (int64_t i = a; i < b; i++) {
            if (sb[i] == (uint8_t)T) {
                snprintf(g_err, sizeof g_err, "string %lld contains the terminator byte 0x%02x",
                         (long long)k, T);
                return OR_E_TERMINATOR;
            }
        }
        int p = 0;
        for (int64_t i = a; i < b; i++) {
            p = ptrie_child_or_add(t, p, sb[i]);
            if (p < 0) return OR_E_NOMEM;
        }
        p = ptrie_child_or_add(t, p, (uint8_t)T);
        if (p < 0) return OR_E_NOMEM;
    }
    /* explicit-stack DFS: pop a node, give it the next id, push its children in
     * descending byte order so the smallest byte is visited first */
    int *order = (int *)malloc((size_t)t->n * sizeof(int));
    int *stack = (int *)malloc((size_t)t->n * sizeof(int));
    if (!order || !stack) {
        free(order);
        free(stack);
        return OR_E_NOMEM;
    }
    int sp = 0, next = 0;
    stack[sp++] = 0;
    while (sp > 0) {
        int p = stack[--sp];
        order[next++] = p;
        const pnode *nd = &t->v[p];
        for (int i = nd->nchild - 1; i >= 0; i--) stack[sp++] = nd->cnode[i];
    }
    free(stack);
    *order_out = order;
    return OR_OK;
}

/*
 * oracle_build: strings in CSR form (bytes str_bytes, offsets str_off[K+1]);
 * set_off[S+1] splits them into S sets (NULL = one set of all K strings).
 * Every set must be non-empty.  terminator in 0..255.
 */
int oracle_build(const uint8_t *str_bytes, const int64_t *str_off, int64_t K,
                 const int64_t *set_off, int64_t S, int terminator, oracle **out) {
    *out = NULL;
    g_err[0] = 0;
    if (K <= 0 || !str_off || (!str_bytes && str_off[K] > 0) || terminator < 0 || terminator > 255) {
        snprintf(g_err, sizeof g_err, "invalid arguments");
        return OR_E_INVAL;
    }
    int64_t one_set[2] = {0, K};
    if (!set_off) {
        set_off = one_set;
        S = 1;
    }
    if (S <= 0 || set_off[0] != 0 || set_off[S] != K) {
        snprintf(g_err, sizeof g_err, "invalid set offsets");
        return OR_E_INVAL;
    }
    for (int64_t j = 0; j < S; j++)
        if (set_off[j + 1] <= set_off[j]) {
            snprintf(g_err, sizeof g_err, "set %lld is empty", (long long)j);
            return OR_E_INVAL;
        }

    oracle *o = (oracle *)calloc(1, sizeof(oracle));
    if (!o) return OR_E_NOMEM;
    o->S = S;
    o->terminator = terminator;
    o->roots = (int32_t *)malloc((size_t)S * sizeof(int32_t));
    int64_t cap = 0, N = 0, E = 0;
    int rc = OR_OK;
    for (int64_t j = 0; j < S && rc == OR_OK; j++) {
        ptrie t;
        int *order = NULL;
        rc = build_set(str_bytes, str_off, set_off[j], set_off[j + 1], terminator, &t, &order);
        if (rc != OR_OK) {
            ptrie_free(&t);
            break;
        }
        int n = t.n;
        if (N + n > cap) {
            int64_t nc = cap ? cap : 1024;
            while (nc < N + n) nc *= 2;
            o->parent = (int32_t *)realloc(o->parent, (size_t)nc * sizeof(int32_t));
            o->depth = (int32_t *)realloc(o->depth, (size_t)nc * sizeof(int32_t));
            o->edge = (uint8_t *)realloc(o->edge, (size_t)nc);
            o->is_final = (uint8_t *)realloc(o->is_final, (size_t)nc);
            o->kid_off = (int64_t *)realloc(o->kid_off, (size_t)(nc + 1) * sizeof(int64_t));
            o->kid_byte = (uint8_t *)realloc(o->kid_byte, (size_t)nc);
            o->kid_node = (int32_t *)realloc(o->kid_node, (size_t)nc * sizeof(int32_t));
            cap = nc;
            if (!o->parent || !o->depth || !o->edge || !o->is_final || !o->kid_off ||
                !o->kid_byte || !o->kid_node) {
                rc = OR_E_NOMEM;
                free(order);
                ptrie_free(&t);
                break;
            }
        }
        /* new id of every pointer node */
        int *newid = (int *)malloc((size_t)n * sizeof(int));
        for (int r = 0; r < n; r++) newid[order[r]] = (int)(N + r);
        o->roots[j] = (int32_t)N;
        o->parent[N] = -1;
        o->depth[N] = 0;
        o->edge[N] = 0;
        o->is_final[N] = 0;
        for (int r = 0; r < n; r++) {
            int p = order[r];
            int64_t id = N + r;
            const pnode *nd = &t.v[p];
            o->kid_off[id] = E;
            for (int i = 0; i < nd->nchild; i++) {
                int64_t c = newid[nd->cnode[i]];
                o->kid_byte[E] = nd->cbyte[i];
                o->kid_node[E] = (int32_t)c;
                E++;
                o->parent[c] = (int32_t)id;
                o->depth[c] = o->depth[id] + 1;
                o->edge[c] = nd->cbyte[i];
                o->is_final[c] = (nd->cbyte[i] == (uint8_t)terminator);
            }
        }
        N += n;
        o->kid_off[N] = E;
        free(newid);
        free(order);
        ptrie_free(&t);
    }
    if (rc != OR_OK) {
        oracle_free(o);
        return rc;
    }
    o->N = N;
    *out = o;
    return OR_OK;
}

int64_t oracle_num_nodes(const oracle *o) { return o->N; }
int64_t oracle_num_sets(const oracle *o) { return o->S; }

void oracle_roots(const oracle *o, int32_t *roots) {
    memcpy(roots, o->roots, (size_t)o->S * sizeof(int32_t));
}

/* Per-node tables in preorder: parent (-1 at a root), depth, the byte on the
 * edge into the node, and whether the node is final (reached by T). */
void oracle_node_info(const oracle *o, int32_t *parent, int32_t *depth, uint8_t *edge,
                      uint8_t *is_final) {
    memcpy(parent, o->parent, (size_t)o->N * sizeof(int32_t));
    memcpy(depth, o->depth, (size_t)o->N * sizeof(int32_t));
    memcpy(edge, o->edge, (size_t)o->N);
    memcpy(is_final, o->is_final, (size_t)o->N);
}

/* ----------------------------------------------------------------- walk --- */

/* delta(n, c): the child of n along byte c, or -1 (dead). */
static int64_t delta(const oracle *o, int64_t n, uint8_t c) {
    for (int64_t i = o->kid_off[n]; i < o->kid_off[n + 1]; i++)
        if (o->kid_byte[i] == c) return o->kid_node[i];
    return -1;
}

/* delta*(n, t): the transition function extended over the bytes of token t
 * (Section 2); -1 once the walk leaves the trie, for an empty token, or for a
 * node outside [0, N). */
static int64_t walk(const oracle *o, int64_t n, const uint8_t *t, int64_t len) {
    if (n < 0 || n >= o->N || len <= 0) return -1;
    for (int64_t i = 0; i < len && n >= 0; i++) n = delta(o, n, t[i]);
    return n;
}

/*
 * Mask rows of the requested nodes (the naive precomputation: every token is
 * walked from the node): out[r*W + (v>>6)] bit (v&63) = walk(node r, t_v) != -1.
 */
int oracle_mask_rows(const oracle *o, const uint8_t *tok_bytes, const int64_t *tok_off, int64_t V,
                     const int32_t *nodes, int64_t n, uint64_t *out) {
    if (V <= 0 || !tok_off || !nodes || !out) return OR_E_INVAL;
    int64_t W = (V + 63) / 64;
    for (int64_t r = 0; r < n; r++) {
        uint64_t *row = out + r * W;
        memset(row, 0, (size_t)W * sizeof(uint64_t));
        for (int64_t v = 0; v < V; v++) {
            if (walk(o, nodes[r], tok_bytes + tok_off[v], tok_off[v + 1] - tok_off[v]) >= 0)
                row[v >> 6] |= (uint64_t)1 << (v & 63);
        }
    }
    return OR_OK;
}

/* State advance: out[b] = delta*(nodes[b], t_{tokens[b]}); -1 when dead or out of range. */
int oracle_advance(const oracle *o, const uint8_t *tok_bytes, const int64_t *tok_off, int64_t V,
                   const int32_t *nodes, const int32_t *tokens, int64_t B, int32_t *out) {
    for (int64_t b = 0; b < B; b++) {
        int64_t v = tokens[b];
        if (v < 0 || v >= V) {
            out[b] = -1;
            continue;
        }
        out[b] = (int32_t)walk(o, nodes[b], tok_bytes + tok_off[v], tok_off[v + 1] - tok_off[v]);
    }
    return OR_OK;
}

/*
 * Apply (Eq. 1 with the mask): logits is B rows of `stride` elements
 * (dtype 0 = fp32, 1 = bf16), row b masked by node nodes[b].  Every token whose
 * walk dies gets the -inf bit pattern; valid entries are left untouched.
 */
int oracle_apply(const oracle *o, const uint8_t *tok_bytes, const int64_t *tok_off, int64_t V,
                 const int32_t *nodes, int64_t B, void *logits, int64_t stride, int dtype) {
    if (dtype != 0 && dtype != 1) return OR_E_INVAL;
    for (int64_t b = 0; b < B; b++) {
        for (int64_t v = 0; v < V; v++) {
            int ok = walk(o, nodes[b], tok_bytes + tok_off[v], tok_off[v + 1] - tok_off[v]) >= 0;
            if (ok) continue;
            if (dtype == 0)
                ((uint32_t *)logits)[b * stride + v] = 0xFF800000u;
            else
                ((uint16_t *)logits)[b * stride + v] = 0xFF80u;
        }
    }
    return OR_OK;
}

/* ------------------------------------------------- fixed-format strings --- */

/*
 * Character-position masks (appendix "Constraint-Aware Dispatch Beyond Finite
 * Sets"): a value of a fixed format has L characters, and character p may be
 * any byte of the class C_p; the value is then closed by the terminator T, as
 * the set strings are.  The states are the positions 0..L (p characters
 * written) and L+1 (after T, final).  Token v is valid at position p iff it is
 * non-empty, p + |t| <= L + 1, and every t[i] lies in C_{p+i}, with C_L = {T};
 * the advance moves to p + |t|, or to the dead state.  A position outside
 * 0..L+1 is dead.
 *
 * classes: L rows of 32 bytes; byte c is in C_p iff bit (c & 7) of
 * classes[32 p + (c >> 3)] is set.
 */
static int fmt_valid(const uint8_t *classes, int64_t L, int T, int64_t p, const uint8_t *t, int64_t len) {
    if (len <= 0 || p < 0 || p + len > L + 1) return 0;
    for (int64_t i = 0; i < len; i++) {
        const int64_t q = p + i;
        const uint8_t c = t[i];
        if (q == L) {
            if (c != (uint8_t)T) return 0;
        } else if (!((classes[q * 32 + (c >> 3)] >> (c & 7)) & 1)) {
            return 0;
        }
    }
    return 1;
}

/* Mask rows of the requested positions, one token at a time. */
int oracle_format_rows(const uint8_t *classes, int64_t L, int T, const uint8_t *tok_bytes,
                       const int64_t *tok_off, int64_t V, const int32_t *pos, int64_t n, uint64_t *out) {
    if (V <= 0 || L < 0 || !tok_off || !pos || !out) return OR_E_INVAL;
    int64_t W = (V + 63) / 64;
    for (int64_t r = 0; r < n; r++) {
        uint64_t *row = out + r * W;
        memset(row, 0, (size_t)W * sizeof(uint64_t));
        for (int64_t v = 0; v < V; v++)
            if (fmt_valid(classes, L, T, pos[r], tok_bytes + tok_off[v], tok_off[v + 1] - tok_off[v]))
                row[v >> 6] |= (uint64_t)1 << (v & 63);
    }
    return OR_OK;
}

/* Advance: out[b] = pos[b] + |t| when token tokens[b] is valid there, else -1. */
int oracle_format_advance(const uint8_t *classes, int64_t L, int T, const uint8_t *tok_bytes,
                          const int64_t *tok_off, int64_t V, const int32_t *pos, const int32_t *tokens,
                          int64_t B, int32_t *out) {
    for (int64_t b = 0; b < B; b++) {
        const int64_t v = tokens[b];
        out[b] = -1;
        if (v < 0 || v >= V) continue;
        const int64_t len = tok_off[v + 1] - tok_off[v];
        if (fmt_valid(classes, L, T, pos[b], tok_bytes + tok_off[v], len)) out[b] = (int32_t)(pos[b] + len);
    }
    return OR_OK;
}
