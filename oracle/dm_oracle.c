/*
 * DualMap routing oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded CPU model of the batched dual-mapping routing
 * path of DualMap (arXiv 2602.06502): chained per-block prefix hashes under two
 * hash functions, two consistent-hash rings, longest cached prefix per
 * candidate, the integer TTFT estimate, the SLO-aware selection with in-order
 * load updates, hotspot-aware rebalancing, and ring scaling with a remap check.
 *
 * Only the test suite, the package's smoke check and the benchmark's CPU
 * baseline load this file's library.  The HIP product path never links, calls
 * or includes it, and the two share no code, headers, tables or constants
 * generators.
 *
 * Each function cites the passage of the paper it follows.  Where the paper is
 * silent (the concrete hash functions, ring point placement, tie-breaking,
 * rounding), the reading taken is stated at the function.  Index membership is
 * deliberately kept as sorted arrays searched by bisection, a different data
 * structure from the device's open-addressing tables.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { OR_OK = 0, OR_EINVAL = 1, OR_ENOMEM = 2, OR_EFULL = 3, OR_ESTATE = 4 };

typedef struct {
    uint32_t block_size;      /* B tokens per KV block (even)                  */
    uint32_t key_blocks;      /* K: ring key covers the first K full blocks     */
    uint64_t seed[2];         /* seeds of f1 and f2                             */
    uint32_t vnodes;          /* V virtual nodes per instance on each ring      */
    uint32_t max_slots;       /* instance ids are < max_slots                   */
    int64_t ttft_base_us;     /* TTFT = base + per_token * uncached             */
    int64_t ttft_per_token_us;/*        + floor(load / queue_div)               */
    int64_t queue_div;
    int64_t slo_us;
} or_config;

typedef struct {
    uint64_t pos;
    uint32_t id;
} or_vnode;

typedef struct {
    or_config cfg;
    uint32_t *kk[2];          /* per-function NH key words, B each (S1)         */
    uint64_t mult[2];         /* per-function chain multiplier P_s              */
    uint64_t h_init[2];       /* per-function chain start H_s[-1]               */
    uint8_t *live;            /* [max_slots] live flags                         */
    uint32_t n_live;
    or_vnode *ring[2];
    uint64_t ring_len;
    uint64_t **set;           /* per instance: sorted unique cached block keys  */
    uint64_t *set_len;
    int policy;               /* selection rule, OR_POLICY_* (default SLO-aware)*/
    /* KV save with LRU eviction: per instance, the keys saved through
     * or_kv_save and the time of their latest touch, sorted by key       */
    uint64_t **lru_key, **lru_t;
    uint64_t *lru_len;
    /* adaptive hash-key length (Sec. 3.2): the prefix hotness tree      */
    int kl_on;
    uint64_t kl_max;          /* most extended prefixes the tree may hold       */
    uint64_t *kl_ext;         /* sorted canon keys of the extended prefixes     */
    uint64_t kl_n;
    uint64_t *kl_log;         /* prefixes (depth >= K) of this window's requests*/
    uint64_t kl_log_n, kl_log_cap;
    uint64_t kl_win;          /* requests routed in this window                 */
} or_state;

/* Selection rules between the two candidates: DualMap's SLO-aware rule and
 * the single-criterion variants of the ablation study (Sec. 4.3). */
enum { OR_POLICY_SLO_AWARE = 0, OR_POLICY_CACHE_AFFINITY = 1, OR_POLICY_LEAST_LOADED = 2,
       OR_POLICY_MIN_TTFT = 3 };

/* ------------------------------------------------------------------------- */
/* Hash primitives.  The paper asks for two independent hash functions over   */
/* the prompt prefix (Sec. 1 and Sec. 3.2) and names none.  The reading taken */
/* here: SplitMix64's finaliser and step (Steele, Lea and Flood, OOPSLA 2014) */
/* with the public-domain splitmix64 constants, NH block digests (Black et    */
/* al., UMAC, CRYPTO 1999) and an affine chain over blocks.                   */
/* ------------------------------------------------------------------------- */

#define OR_GOLDEN 0x9E3779B97F4A7C15ULL

uint64_t or_mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

static uint64_t sm_next(uint64_t *state)
{
    *state += OR_GOLDEN;
    return or_mix64(*state);
}

/* Per-function parameters drawn from a SplitMix64 stream started at the
 * function's seed: B key words, then the (odd) chain multiplier, then the
 * chain's start value. */
void or_params(uint64_t seed, uint32_t B, uint32_t *kk, uint64_t *mult, uint64_t *h_init)
{
    uint64_t st = seed;
    for (uint32_t j = 0; j < B; j++)
        kk[j] = (uint32_t)sm_next(&st);
    *mult = sm_next(&st) | 1ULL;
    *h_init = sm_next(&st);
}

/* NH digest of one block of B tokens: the sum over token pairs of the product
 * of the two 32-bit sums (token + key word), taken modulo 2^64. */
uint64_t or_nh(const int32_t *t, const uint32_t *kk, uint32_t B)
{
    uint64_t acc = 0;
    for (uint32_t j = 0; j + 1 < B; j += 2) {
        uint32_t a = (uint32_t)t[j] + kk[j];
        uint32_t b = (uint32_t)t[j + 1] + kk[j + 1];
        acc += (uint64_t)a * (uint64_t)b;
    }
    return acc;
}

/* Chained per-block prefix hash of one prompt under function s (KV metadata
 * keeps one hash per block, Sec. A.3.2 "Metadata footprint").  The chain value
 * after block b is H[b] = H[b-1] * P + NH(b); the block key is
 * mix64(H[b] xor seed).  Only full blocks are hashed; trailing tokens that do
 * not fill a block are not.  Writes nfull keys to out (if not NULL) and
 * returns nfull. */
uint64_t or_chain(const or_state *st, int s, const int32_t *t, int64_t len, uint64_t *out)
{
    const uint32_t B = st->cfg.block_size;
    const uint64_t nfull = len > 0 ? (uint64_t)len / B : 0;
    uint64_t H = st->h_init[s];
    for (uint64_t b = 0; b < nfull; b++) {
        H = H * st->mult[s] + or_nh(t + b * B, st->kk[s], B);
        if (out)
            out[b] = or_mix64(H ^ st->cfg.seed[s]);
    }
    return nfull;
}

/* Ring key of a prompt under function s (dual mapping, Sec. 3.2 and
 * Sec. A.7): the block key of the last block of the hashed prefix, which is
 * the first K full blocks (fewer if the prompt is shorter).  A prompt with no
 * full block maps to the key of the empty prefix, mix64(H[-1] xor seed). */
uint64_t or_ring_key_at(const or_state *st, int s, const int32_t *t, uint64_t kr);

uint64_t or_ring_key(const or_state *st, int s, const int32_t *t, int64_t len)
{
    const uint32_t B = st->cfg.block_size;
    uint64_t nfull = len > 0 ? (uint64_t)len / B : 0;
    uint64_t kr = nfull < st->cfg.key_blocks ? nfull : st->cfg.key_blocks;
    return or_ring_key_at(st, s, t, kr);
}

/* Ring key of the first kr full blocks under function s (kr = 0: the
 * empty-prefix key).  The prompt must hold kr full blocks. */
uint64_t or_ring_key_at(const or_state *st, int s, const int32_t *t, uint64_t kr)
{
    const uint32_t B = st->cfg.block_size;
    uint64_t H = st->h_init[s];
    for (uint64_t b = 0; b < kr; b++)
        H = H * st->mult[s] + or_nh(t + b * B, st->kk[s], B);
    return or_mix64(H ^ st->cfg.seed[s]);
}

/* Ring position of virtual node v of instance id on ring s.  The paper gives
 * each instance one anchor derived from a unique identifier (Sec. 3.4); the
 * reading taken adds V virtual nodes per instance, placed by a bijective mix
 * of (id, v) so positions never tie within a ring and do not depend on which
 * other instances are live. */
uint64_t or_vpos(const or_state *st, int s, uint32_t id, uint32_t v)
{
    return or_mix64((((uint64_t)id << 32) | v) ^ or_mix64(st->cfg.seed[s]));
}

/* Successor rule of the ring (Sec. A.1.3, worked example (A,B] -> B): the
 * owner of position x is the first ring entry at a position >= x, wrapping to
 * the first entry when x lies past the last one.  pos must be ascending. */
uint32_t or_owner_sorted(const uint64_t *pos, const uint32_t *id, uint64_t len, uint64_t x)
{
    uint64_t lo = 0, hi = len; /* first index with pos >= x */
    while (lo < hi) {
        uint64_t mid = lo + (hi - lo) / 2;
        if (pos[mid] < x)
            lo = mid + 1;
        else
            hi = mid;
    }
    return id[lo == len ? 0 : lo];
}

static uint32_t ring_owner(const or_state *st, int s, uint64_t x)
{
    const or_vnode *r = st->ring[s];
    uint64_t lo = 0, hi = st->ring_len;
    while (lo < hi) {
        uint64_t mid = lo + (hi - lo) / 2;
        if (r[mid].pos < x)
            lo = mid + 1;
        else
            hi = mid;
    }
    return r[lo == st->ring_len ? 0 : lo].id;
}

uint32_t or_owner(const or_state *st, int s, uint64_t x)
{
    if (!st || st->ring_len == 0 || s < 0 || s > 1)
        return 0xFFFFFFFFu;
    return ring_owner(st, s, x);
}

/* ------------------------------------------------------------------------- */
/* Sorting (a library-style primitive: LSD radix sort of u64 keys).           */
/* ------------------------------------------------------------------------- */

static int sort_u64(uint64_t *a, uint64_t n)
{
    if (n < 2)
        return OR_OK;
    uint64_t *tmp = (uint64_t *)malloc(n * sizeof(uint64_t));
    if (!tmp)
        return OR_ENOMEM;
    uint64_t *src = a, *dst = tmp;
    for (int shift = 0; shift < 64; shift += 8) {
        uint64_t count[257] = {0};
        for (uint64_t i = 0; i < n; i++)
            count[((src[i] >> shift) & 0xFF) + 1]++;
        for (int d = 0; d < 256; d++)
            count[d + 1] += count[d];
        for (uint64_t i = 0; i < n; i++)
            dst[count[(src[i] >> shift) & 0xFF]++] = src[i];
        uint64_t *sw = src; src = dst; dst = sw;
    }
    /* eight passes: the sorted data is back in a */
    free(tmp);
    return OR_OK;
}

int or_sort_u64(uint64_t *a, uint64_t n) { return sort_u64(a, n); }

static int cmp_vnode(const void *pa, const void *pb)
{
    const or_vnode *a = (const or_vnode *)pa, *b = (const or_vnode *)pb;
    if (a->pos != b->pos)
        return a->pos < b->pos ? -1 : 1;
    return a->id < b->id ? -1 : (a->id > b->id ? 1 : 0);
}

/* ------------------------------------------------------------------------- */
/* State                                                                     */
/* ------------------------------------------------------------------------- */

or_state *or_create(const or_config *cfg)
{
    if (!cfg || cfg->block_size < 2 || (cfg->block_size & 1) || cfg->key_blocks < 1 ||
        cfg->vnodes < 1 || cfg->max_slots < 1 || cfg->queue_div < 1)
        return NULL;
    or_state *st = (or_state *)calloc(1, sizeof(or_state));
    if (!st)
        return NULL;
    st->cfg = *cfg;
    for (int s = 0; s < 2; s++) {
        st->kk[s] = (uint32_t *)malloc(cfg->block_size * sizeof(uint32_t));
        if (!st->kk[s])
            goto fail;
        or_params(cfg->seed[s], cfg->block_size, st->kk[s], &st->mult[s], &st->h_init[s]);
    }
    st->live = (uint8_t *)calloc(cfg->max_slots, 1);
    st->set = (uint64_t **)calloc(cfg->max_slots, sizeof(uint64_t *));
    st->set_len = (uint64_t *)calloc(cfg->max_slots, sizeof(uint64_t));
    st->lru_key = (uint64_t **)calloc(cfg->max_slots, sizeof(uint64_t *));
    st->lru_t = (uint64_t **)calloc(cfg->max_slots, sizeof(uint64_t *));
    st->lru_len = (uint64_t *)calloc(cfg->max_slots, sizeof(uint64_t));
    if (!st->live || !st->set || !st->set_len || !st->lru_key || !st->lru_t || !st->lru_len)
        goto fail;
    return st;
fail:
    free(st->kk[0]); free(st->kk[1]); free(st->live); free(st->set); free(st->set_len);
    free(st->lru_key); free(st->lru_t); free(st->lru_len);
    free(st);
    return NULL;
}

void or_destroy(or_state *st)
{
    if (!st)
        return;
    free(st->kl_ext);
    free(st->kl_log);
    for (uint32_t i = 0; i < st->cfg.max_slots; i++) {
        free(st->set[i]);
        free(st->lru_key[i]);
        free(st->lru_t[i]);
    }
    free(st->set); free(st->set_len); free(st->live);
    free(st->lru_key); free(st->lru_t); free(st->lru_len);
    free(st->ring[0]); free(st->ring[1]);
    free(st->kk[0]); free(st->kk[1]);
    free(st);
}

/* Build both rings for the live flags currently in st->live. */
static int rebuild_rings(or_state *st)
{
    uint64_t len = (uint64_t)st->n_live * st->cfg.vnodes;
    or_vnode *r[2] = {NULL, NULL};
    for (int s = 0; s < 2; s++) {
        r[s] = (or_vnode *)malloc((len ? len : 1) * sizeof(or_vnode));
        if (!r[s]) {
            free(r[0]);
            return OR_ENOMEM;
        }
        uint64_t k = 0;
        for (uint32_t id = 0; id < st->cfg.max_slots; id++) {
            if (!st->live[id])
                continue;
            for (uint32_t v = 0; v < st->cfg.vnodes; v++) {
                r[s][k].pos = or_vpos(st, s, id, v);
                r[s][k].id = id;
                k++;
            }
        }
        qsort(r[s], len, sizeof(or_vnode), cmp_vnode);
    }
    free(st->ring[0]); free(st->ring[1]);
    st->ring[0] = r[0];
    st->ring[1] = r[1];
    st->ring_len = len;
    return OR_OK;
}

/* Initial membership: the live set is exactly ids[0..n). */
int or_build_rings(or_state *st, const uint32_t *ids, uint32_t n)
{
    if (!st || (!ids && n) || n == 0)
        return OR_EINVAL;
    uint8_t *seen = (uint8_t *)calloc(st->cfg.max_slots, 1);
    if (!seen)
        return OR_ENOMEM;
    for (uint32_t i = 0; i < n; i++) {
        if (ids[i] >= st->cfg.max_slots || seen[ids[i]]) {
            free(seen);
            return OR_EINVAL;
        }
        seen[ids[i]] = 1;
    }
    memcpy(st->live, seen, st->cfg.max_slots);
    free(seen);
    st->n_live = n;
    return rebuild_rings(st);
}

/* Copy of the ring arrays (for tests). */
uint64_t or_ring_copy(const or_state *st, int s, uint64_t *pos, uint32_t *id)
{
    if (!st || s < 0 || s > 1)
        return 0;
    for (uint64_t i = 0; i < st->ring_len; i++) {
        if (pos) pos[i] = st->ring[s][i].pos;
        if (id) id[i] = st->ring[s][i].id;
    }
    return st->ring_len;
}

/* Index keys avoid the two reserved values 0 and 1 by moving them to
 * 2^63 and 2^63 + 1 (a reading of this build; the paper stores one 8-byte
 * hash per block, Sec. A.3.2). */
static uint64_t canon(uint64_t k) { return k >= 2 ? k : k + (1ULL << 63); }

uint64_t or_canon(uint64_t k) { return canon(k); }

static int set_contains(const or_state *st, uint32_t id, uint64_t key)
{
    const uint64_t *a = st->set[id];
    uint64_t lo = 0, hi = st->set_len[id];
    while (lo < hi) {
        uint64_t mid = lo + (hi - lo) / 2;
        if (a[mid] < key)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo < st->set_len[id] && a[lo] == key;
}

int or_index_contains(const or_state *st, uint32_t id, uint64_t key)
{
    if (!st || id >= st->cfg.max_slots)
        return 0;
    return set_contains(st, id, canon(key));
}

/* Add keys to instance id's cached block set (set semantics). */
int or_index_insert(or_state *st, uint32_t id, const uint64_t *keys, uint64_t n)
{
    if (!st || id >= st->cfg.max_slots || (!keys && n))
        return OR_EINVAL;
    if (n == 0)
        return OR_OK;
    uint64_t old = st->set_len[id];
    uint64_t *a = (uint64_t *)realloc(st->set[id], (old + n) * sizeof(uint64_t));
    if (!a)
        return OR_ENOMEM;
    for (uint64_t i = 0; i < n; i++)
        a[old + i] = canon(keys[i]);
    if (sort_u64(a, old + n) != OR_OK)
        return OR_ENOMEM;
    uint64_t w = 0;
    for (uint64_t i = 0; i < old + n; i++)
        if (w == 0 || a[i] != a[w - 1])
            a[w++] = a[i];
    st->set[id] = a;
    st->set_len[id] = w;
    return OR_OK;
}

int or_index_erase(or_state *st, uint32_t id, const uint64_t *keys, uint64_t n)
{
    if (!st || id >= st->cfg.max_slots || (!keys && n))
        return OR_EINVAL;
    uint64_t *a = st->set[id];
    uint64_t len = st->set_len[id];
    if (n == 0 || len == 0)
        return OR_OK;
    /* mark every present key, then keep the unmarked ones in order */
    uint8_t *gone = (uint8_t *)calloc(len, 1);
    if (!gone)
        return OR_ENOMEM;
    for (uint64_t i = 0; i < n; i++) {
        uint64_t k = canon(keys[i]);
        uint64_t lo = 0, hi = len;
        while (lo < hi) {
            uint64_t mid = lo + (hi - lo) / 2;
            if (a[mid] < k) lo = mid + 1; else hi = mid;
        }
        if (lo < len && a[lo] == k)
            gone[lo] = 1;
    }
    uint64_t w = 0;
    for (uint64_t i = 0; i < len; i++)
        if (!gone[i])
            a[w++] = a[i];
    free(gone);
    st->set_len[id] = w;
    return OR_OK;
}

int or_index_clear(or_state *st, uint32_t id)
{
    if (!st || id >= st->cfg.max_slots)
        return OR_EINVAL;
    free(st->set[id]);
    st->set[id] = NULL;
    st->set_len[id] = 0;
    free(st->lru_key[id]); st->lru_key[id] = NULL;
    free(st->lru_t[id]); st->lru_t[id] = NULL;
    st->lru_len[id] = 0;
    return OR_OK;
}

uint64_t or_index_size(const or_state *st, uint32_t id)
{
    return (st && id < st->cfg.max_slots) ? st->set_len[id] : 0;
}

/* ------------------------------------------------------------------------- */
/* KV save with least-recently-used eviction: the step after routing.  A     */
/* served request's KV blocks are saved on its instance (the KV query and   */
/* save of Sec. A.3.2), and each instance's cache is bounded.               */
/* ------------------------------------------------------------------------- */

typedef struct {
    uint64_t key, t;
} or_kt;

static int cmp_kt_key(const void *pa, const void *pb)
{
    const or_kt *a = (const or_kt *)pa, *b = (const or_kt *)pb;
    if (a->key != b->key)
        return a->key < b->key ? -1 : 1;
    return a->t > b->t ? -1 : (a->t < b->t ? 1 : 0); /* latest touch first */
}

static int cmp_kt_time_desc(const void *pa, const void *pb)
{
    const or_kt *a = (const or_kt *)pa, *b = (const or_kt *)pb;
    return a->t > b->t ? -1 : (a->t < b->t ? 1 : 0);
}

/* Save the batch's blocks: request r (full blocks block_keys[start_r ..
 * start_r + nfull_r), request-major, start_r = full blocks of the requests
 * before it) is served by inst[r].  Every block is touched on that
 * instance, deepest block first, at time clock + start_r + (nfull_r - 1 - b)
 * for block b, so a prefix's blocks are always more recent than its
 * descendants.  Each instance's cache becomes the cap most recently touched
 * distinct keys (cap = 0: unbounded) among what it held and what it was
 * sent; keys that leave are erased from its index and keys that join are
 * inserted.  *added and *removed (optional) count them over all instances.
 * The caller's clock should advance by the batch's full blocks. */
int or_kv_save(or_state *st, const int64_t *off, uint64_t n, const uint64_t *block_keys,
               const uint32_t *inst, uint64_t clock, uint64_t cap, uint64_t *added,
               uint64_t *removed)
{
    if (!st || (n && (!off || !inst)))
        return OR_EINVAL;
    const uint32_t S = st->cfg.max_slots, B = st->cfg.block_size;
    uint64_t total = 0;
    for (uint64_t r = 0; r < n; r++) {
        if (off[r + 1] < off[r] || inst[r] >= S)
            return OR_EINVAL;
        total += (uint64_t)(off[r + 1] - off[r]) / B;
    }
    if (total && !block_keys)
        return OR_EINVAL;
    /* every block's (instance, key, time), grouped by instance */
    uint64_t *cnt = (uint64_t *)calloc(S + 1, sizeof(uint64_t));
    or_kt *ent = (or_kt *)malloc((total ? total : 1) * sizeof(or_kt));
    if (!cnt || !ent) {
        free(cnt); free(ent);
        return OR_ENOMEM;
    }
    for (uint64_t r = 0; r < n; r++)
        cnt[inst[r] + 1] += (uint64_t)(off[r + 1] - off[r]) / B;
    for (uint32_t c = 0; c < S; c++)
        cnt[c + 1] += cnt[c];
    uint64_t start = 0;
    for (uint64_t r = 0; r < n; r++) {
        const uint64_t nf = (uint64_t)(off[r + 1] - off[r]) / B;
        for (uint64_t b = 0; b < nf; b++) {
            or_kt *e = &ent[cnt[inst[r]]++];
            e->key = block_keys[start + b];
            e->t = clock + start + (nf - 1 - b);
        }
        start += nf;
    }
    /* cnt[c] is now the end of instance c's entries; its start is cnt[c-1] */
    uint64_t n_add = 0, n_rm = 0;
    int rc = OR_OK;
    for (uint32_t c = 0; c < S && rc == OR_OK; c++) {
        const uint64_t lo = c ? cnt[c - 1] : 0, hi = cnt[c];
        /* an instance sent nothing still keeps only its cap most recent keys */
        if (lo == hi && (cap == 0 || st->lru_len[c] <= cap))
            continue;
        const uint64_t old = st->lru_len[c], m = old + (hi - lo);
        or_kt *a = (or_kt *)malloc(m * sizeof(or_kt));
        uint64_t *gone = (uint64_t *)malloc((old ? old : 1) * sizeof(uint64_t));
        uint64_t *join = (uint64_t *)malloc(m * sizeof(uint64_t));
        if (!a || !gone || !join) {
            free(a); free(gone); free(join);
            rc = OR_ENOMEM;
            break;
        }
        for (uint64_t k = 0; k < old; k++) {
            a[k].key = st->lru_key[c][k];
            a[k].t = st->lru_t[c][k];
        }
        memcpy(a + old, ent + lo, (hi - lo) * sizeof(or_kt));
        /* latest touch per key */
        qsort(a, m, sizeof(or_kt), cmp_kt_key);
        uint64_t u = 0;
        for (uint64_t k = 0; k < m; k++)
            if (u == 0 || a[k].key != a[u - 1].key)
                a[u++] = a[k];
        /* the cap most recent keys stay */
        if (cap && u > cap) {
            qsort(a, u, sizeof(or_kt), cmp_kt_time_desc);
            u = cap;
            qsort(a, u, sizeof(or_kt), cmp_kt_key);
        }
        /* keys that left and keys that joined (both lists sorted by key) */
        uint64_t ng = 0, nj = 0, i = 0, j = 0;
        while (i < old || j < u) {
            if (j == u || (i < old && st->lru_key[c][i] < a[j].key))
                gone[ng++] = st->lru_key[c][i++];
            else if (i == old || a[j].key < st->lru_key[c][i])
                join[nj++] = a[j++].key;
            else {
                i++;
                j++;
            }
        }
        if (or_index_erase(st, c, gone, ng) != OR_OK || or_index_insert(st, c, join, nj) != OR_OK)
            rc = OR_ENOMEM;
        uint64_t *nk = (uint64_t *)realloc(st->lru_key[c], (u ? u : 1) * sizeof(uint64_t));
        uint64_t *nt = nk ? (uint64_t *)realloc(st->lru_t[c], (u ? u : 1) * sizeof(uint64_t)) : NULL;
        if (!nk || !nt) {
            if (nk) st->lru_key[c] = nk;
            free(a); free(gone); free(join);
            rc = OR_ENOMEM;
            break;
        }
        for (uint64_t k = 0; k < u; k++) {
            nk[k] = a[k].key;
            nt[k] = a[k].t;
        }
        st->lru_key[c] = nk;
        st->lru_t[c] = nt;
        st->lru_len[c] = u;
        n_add += nj;
        n_rm += ng;
        free(a); free(gone); free(join);
    }
    free(cnt);
    free(ent);
    if (added) *added = n_add;
    if (removed) *removed = n_rm;
    return rc;
}

/* ------------------------------------------------------------------------- */
/* Queued requests: the serving state the rebalancing pass reads (Sec. 3.3). */
/* Per instance a FIFO of records (request id, uncached tokens on it, the    */
/* other candidate, uncached tokens there) in CSR form over instance slots, */
/* and base work ahead of each queue.  Every operation writes a new CSR.    */
/* ------------------------------------------------------------------------- */

/* A routed batch joins the queues: request r (id rec_base + r) at the tail
 * of its chosen instance's queue, in request order; its uncached tokens are
 * len - B * match on each candidate, the other candidate its alternative. */
int or_queue_append(const or_state *st, const int64_t *qoff, const uint64_t *rec,
                    const uint32_t *here, const uint32_t *alt, const uint32_t *there, uint64_t nb,
                    const int64_t *off, const uint32_t *cand, const uint32_t *match,
                    const uint32_t *chosen, uint64_t rec_base, int64_t *qoff2, uint64_t *rec2,
                    uint32_t *here2, uint32_t *alt2, uint32_t *there2)
{
    if (!st || !qoff || !qoff2)
        return OR_EINVAL;
    const uint32_t S = st->cfg.max_slots;
    const int64_t B = st->cfg.block_size;
    for (uint64_t r = 0; r < nb; r++)
        if (chosen[r] >= S || off[r + 1] < off[r])
            return OR_EINVAL;
    qoff2[0] = 0;
    for (uint32_t i = 0; i < S; i++) {
        int64_t w = qoff2[i];
        for (int64_t q = qoff[i]; q < qoff[i + 1]; q++, w++) {
            rec2[w] = rec[q]; here2[w] = here[q]; alt2[w] = alt[q]; there2[w] = there[q];
        }
        for (uint64_t r = 0; r < nb; r++) {
            if (chosen[r] != i)
                continue;
            const int64_t len = off[r + 1] - off[r];
            const uint32_t c1 = cand[r], c2 = cand[nb + r];
            const int64_t u1 = len - B * (int64_t)match[r], u2 = len - B * (int64_t)match[nb + r];
            const int first = chosen[r] == c1;
            rec2[w] = rec_base + r;
            here2[w] = (uint32_t)(first ? u1 : u2);
            alt2[w] = first ? c2 : c1;
            there2[w] = (uint32_t)(first ? u2 : u1);
            w++;
        }
        qoff2[i + 1] = w;
    }
    return OR_OK;
}

/* A migration list applied in order: each record leaves its source queue
 * (the others keep their order) and joins its target's tail with the pair's
 * roles swapped (its alternative becomes the source). */
int or_queue_migrate(const or_state *st, const int64_t *qoff, const uint64_t *rec,
                     const uint32_t *here, const uint32_t *alt, const uint32_t *there, uint64_t m,
                     const uint64_t *mrec, const uint32_t *msrc, const uint32_t *mdst,
                     int64_t *qoff2, uint64_t *rec2, uint32_t *here2, uint32_t *alt2,
                     uint32_t *there2)
{
    if (!st || !qoff || !qoff2)
        return OR_EINVAL;
    const uint32_t S = st->cfg.max_slots;
    const uint64_t Q = (uint64_t)qoff[S];
    /* the queue position of every migrated record */
    int64_t *at = (int64_t *)malloc((m ? m : 1) * sizeof(int64_t));
    uint8_t *gone = (uint8_t *)calloc(Q ? Q : 1, 1);
    if (!at || !gone) {
        free(at); free(gone);
        return OR_ENOMEM;
    }
    for (uint64_t k = 0; k < m; k++) {
        at[k] = -1;
        if (msrc[k] >= S || mdst[k] >= S) {
            free(at); free(gone);
            return OR_EINVAL;
        }
        for (int64_t q = qoff[msrc[k]]; q < qoff[msrc[k] + 1]; q++)
            if (rec[q] == mrec[k] && !gone[q]) {
                at[k] = q;
                gone[q] = 1;
                break;
            }
        if (at[k] < 0) {
            free(at); free(gone);
            return OR_EINVAL;
        }
    }
    qoff2[0] = 0;
    for (uint32_t i = 0; i < S; i++) {
        int64_t w = qoff2[i];
        for (int64_t q = qoff[i]; q < qoff[i + 1]; q++)
            if (!gone[q]) {
                rec2[w] = rec[q]; here2[w] = here[q]; alt2[w] = alt[q]; there2[w] = there[q];
                w++;
            }
        for (uint64_t k = 0; k < m; k++)
            if (mdst[k] == i) {
                const int64_t q = at[k];
                rec2[w] = rec[q]; here2[w] = there[q]; alt2[w] = msrc[k]; there2[w] = here[q];
                w++;
            }
        qoff2[i + 1] = w;
    }
    free(at);
    free(gone);
    return OR_OK;
}

/* units[i] of service on instance i: base work first, then whole records
 * from the head; a partly served head keeps the remainder. */
int or_queue_drain(const or_state *st, const int64_t *qoff, const uint64_t *rec,
                   const uint32_t *here, const uint32_t *alt, const uint32_t *there,
                   const int64_t *base, const int64_t *units, int64_t *qoff2, uint64_t *rec2,
                   uint32_t *here2, uint32_t *alt2, uint32_t *there2, int64_t *base2)
{
    if (!st || !qoff || !qoff2 || !base || !units || !base2)
        return OR_EINVAL;
    const uint32_t S = st->cfg.max_slots;
    qoff2[0] = 0;
    for (uint32_t i = 0; i < S; i++) {
        if (units[i] < 0 || base[i] < 0)
            return OR_EINVAL;
        int64_t u = units[i];
        const int64_t take = base[i] < u ? base[i] : u;
        base2[i] = base[i] - take;
        u -= take;
        int64_t q = qoff[i];
        while (q < qoff[i + 1] && u >= (int64_t)here[q]) {
            u -= here[q];
            q++;
        }
        int64_t w = qoff2[i];
        for (int64_t p = q; p < qoff[i + 1]; p++, w++) {
            rec2[w] = rec[p];
            here2[w] = (uint32_t)(p == q ? (int64_t)here[p] - u : (int64_t)here[p]);
            alt2[w] = alt[p];
            there2[w] = there[p];
        }
        qoff2[i + 1] = w;
    }
    return OR_OK;
}

/* ------------------------------------------------------------------------- */
/* Routing                                                                   */
/* ------------------------------------------------------------------------- */

/* Floor division of a (possibly negative) int64 by a positive divisor. */
static int64_t floor_div(int64_t a, int64_t d)
{
    int64_t q = a / d;
    if ((a % d != 0) && (a < 0))
        q -= 1;
    return q;
}

/* Estimated TTFT of a request on an instance: queueing delay plus compute
 * (Sec. 3.2, TTFT(r,i) = T_q(r,i) + T_c(r,i); Sec. A.1.1).  Load is the number
 * of pending prefill tokens (Sec. 3.2).  Integer form taken here:
 * base + per_token * uncached_tokens + floor(load / queue_div) microseconds. */
int64_t or_ttft(const or_state *st, int64_t uncached, int64_t load)
{
    return st->cfg.ttft_base_us + st->cfg.ttft_per_token_us * uncached +
           floor_div(load, st->cfg.queue_div);
}

/* Next live id after c in ascending cyclic id order; with dense ids
 * 0..n-1 this is (c + 1) mod n, the second-candidate adjustment of Sec. 3.2. */
static uint32_t next_live(const or_state *st, uint32_t c)
{
    for (uint32_t step = 1; step <= st->cfg.max_slots; step++) {
        uint32_t id = (uint32_t)(((uint64_t)c + step) % st->cfg.max_slots);
        if (st->live[id])
            return id;
    }
    return c;
}

/* Candidate pair of a request (dual mapping on the dual hash ring,
 * Sec. 3.2 and Sec. 3.4): the owner of each ring key on its ring; if both
 * land on one instance the second becomes the next live instance.  Returns 1
 * if that adjustment was applied (always so when only one instance is
 * live). */
int or_candidates(const or_state *st, uint64_t x1, uint64_t x2, uint32_t *c1, uint32_t *c2)
{
    *c1 = ring_owner(st, 0, x1);
    uint32_t raw2 = ring_owner(st, 1, x2);
    if (raw2 != *c1) {
        *c2 = raw2;
        return 0;
    }
    *c2 = st->n_live >= 2 ? next_live(st, *c1) : *c1;
    return 1;
}

/* Number of leading full blocks of the request whose block keys (f1 chain)
 * are all cached on instance id: the longest cached prefix in blocks
 * ("reusable tokens" of the KV-cache query, Sec. A.3.2). */
static uint64_t prefix_match(const or_state *st, uint32_t id, const uint64_t *h1, uint64_t nfull)
{
    uint64_t m = 0;
    while (m < nfull && set_contains(st, id, canon(h1[m])))
        m++;
    return m;
}

/* Queued records re-priced against the caches as they are now: each TTFT
 * the rebalancing pass evaluates rests on a KV-cache query on the record's
 * instance and one on its backup (Sec. A.3.2, rebalancing cost; Sec. 3.3).
 * Record id r's f1 block chain is keys[coff[r] .. coff[r+1]) and its prompt
 * plen[r] tokens; its uncached tokens become plen - B * (cached leading
 * blocks of the chain) on its instance (here2) and on its alternative
 * (there2).  Order, ids, alternatives and base work are unchanged.
 * OR_EINVAL for an id >= n_ids, a chain with more blocks than the prompt
 * holds, or a prompt outside [0, 2^32). */
int or_queue_reprobe(const or_state *st, const int64_t *qoff, const uint64_t *rec,
                     const uint32_t *alt, uint64_t n_ids, const int64_t *coff,
                     const uint64_t *keys, const int64_t *plen, uint32_t *here2, uint32_t *there2)
{
    if (!st || !qoff)
        return OR_EINVAL;
    const uint32_t S = st->cfg.max_slots;
    const int64_t B = st->cfg.block_size;
    for (uint32_t i = 0; i < S; i++) {
        for (int64_t q = qoff[i]; q < qoff[i + 1]; q++) {
            const uint64_t r = rec[q];
            if (r >= n_ids || alt[q] >= S)
                return OR_EINVAL;
            const int64_t nb = coff[r + 1] - coff[r];
            if (coff[r] < 0 || nb < 0 || plen[r] < 0 || plen[r] >= ((int64_t)1 << 32) ||
                nb * B > plen[r])
                return OR_EINVAL;
            const uint64_t *h1 = keys + coff[r];
            here2[q] = (uint32_t)(plen[r] - B * (int64_t)prefix_match(st, i, h1, (uint64_t)nb));
            there2[q] = (uint32_t)(plen[r] - B * (int64_t)prefix_match(st, alt[q], h1, (uint64_t)nb));
        }
    }
    return OR_OK;
}

/* Selection of one request between its candidates.  Loads L are pending
 * prefill tokens before this request.  SLO-aware rule (Sec. 3.2 "SLO-Aware
 * Strategy"; Sec. A.1.1):
 *   - equal prefix hits: the less-loaded candidate (ties: c1);
 *   - otherwise the candidate with more cached blocks, unless its TTFT
 *     exceeds the SLO, then the less-loaded one (ties: keep the cached one).
 * Ablation variants (Sec. 4.3), each a single criterion:
 *   - cache affinity: the candidate with more cached blocks (equal hits: the
 *     less-loaded, ties c1);
 *   - least loaded: the less-loaded candidate (ties: c1);
 *   - min TTFT: the candidate with the smaller estimated TTFT (ties: c1).
 * Flags: bit0 the chosen candidate has fewer cached blocks than the other
 * (under the SLO-aware rule: a switch for the SLO), bit1 both candidates'
 * TTFT exceed the SLO, bit2 equal match, bit3 the second candidate was
 * adjusted. */
uint32_t or_select(const or_state *st, uint32_t c1, uint32_t c2, uint64_t m1, uint64_t m2,
                   int64_t len, const int64_t *L, int64_t *ttft_out, uint8_t *flags_io)
{
    const int64_t B = st->cfg.block_size;
    const int64_t unc1 = len - B * (int64_t)m1, unc2 = len - B * (int64_t)m2;
    const int64_t t1 = or_ttft(st, unc1, L[c1]), t2 = or_ttft(st, unc2, L[c2]);
    uint8_t fl = *flags_io;
    if (t1 > st->cfg.slo_us && t2 > st->cfg.slo_us)
        fl |= 2;
    if (m1 == m2)
        fl |= 4;
    uint32_t ch;
    switch (st->policy) {
    case OR_POLICY_LEAST_LOADED:
        ch = (L[c1] <= L[c2]) ? c1 : c2;
        break;
    case OR_POLICY_MIN_TTFT:
        ch = (t1 <= t2) ? c1 : c2;
        break;
    case OR_POLICY_CACHE_AFFINITY:
        if (m1 == m2)
            ch = (L[c1] <= L[c2]) ? c1 : c2;
        else
            ch = m1 > m2 ? c1 : c2;
        break;
    default:
        if (m1 == m2) {
            ch = (L[c1] <= L[c2]) ? c1 : c2;
        } else {
            uint32_t a = m1 > m2 ? c1 : c2, o = m1 > m2 ? c2 : c1;
            int64_t ta = m1 > m2 ? t1 : t2;
            if (ta <= st->cfg.slo_us)
                ch = a;
            else if (L[o] < L[a])
                ch = o;
            else
                ch = a;
        }
    }
    if (m1 != m2 && (ch == c1) != (m1 > m2))
        fl |= 1;
    *ttft_out = (ch == c1) ? t1 : t2;
    *flags_io = fl;
    return ch;
}

/* Choose the selection rule for later routes; OR_EINVAL if unknown. */
int or_set_policy(or_state *st, int policy)
{
    if (!st || policy < OR_POLICY_SLO_AWARE || policy > OR_POLICY_MIN_TTFT)
        return OR_EINVAL;
    st->policy = policy;
    return OR_OK;
}

/* ------------------------------------------------------------------------- */
/* Adaptive hash-key length (Sec. 3.2, "How long prefix is appropriate for   */
/* the hash key?"; Sec. A.1.1, Fig. prefix-len).                              */
/* ------------------------------------------------------------------------- */

/* The prefix hotness tree.  A node is a prompt prefix of d >= K full blocks,
 * named by the f1 key of its last block (that key covers the whole prefix);
 * the nodes of depth K are the roots.  The tree is held as the set of its
 * extended nodes, those whose children exist.  A request's hash prefix is
 * its path from its root to a leaf: K_r is the smallest d >= K whose prefix
 * is not extended, and never more than the request's full blocks (fewer
 * than K full blocks: all of them, as without the tree).
 *
 * Traffic ratios come from windows the caller closes (or_keylen_window):
 * rho of a prefix = requests of the window that carry it / requests routed
 * in the window.  At the close, with n live instances, a leaf with
 * rho > 2/n becomes extended (its children are added, so its requests hash
 * one block more and spread over more candidate pairs) and an extended node
 * with rho < 1/n is no longer (its children are removed).  The rule is
 * applied until it changes nothing: a child added as hot that is itself hot
 * in the same window is extended too, so a hot prefix grows in one close to
 * where its requests part.  Since a prefix's count never exceeds its
 * parent's, that fixed point is the set of prefixes (depth >= K) with
 * rho > 2/n, or already extended with rho >= 1/n; it is a tree (every
 * member's parent is a member). */

static int kl_extended(const or_state *st, uint64_t ck)
{
    uint64_t lo = 0, hi = st->kl_n;
    while (lo < hi) {
        uint64_t mid = lo + (hi - lo) / 2;
        if (st->kl_ext[mid] < ck)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo < st->kl_n && st->kl_ext[lo] == ck;
}

/* K_r of a request with block keys h1[0..nfull). */
static uint64_t kl_key_len(const or_state *st, const uint64_t *h1, uint64_t nfull)
{
    const uint64_t K = st->cfg.key_blocks;
    if (nfull <= K || !st->kl_on)
        return nfull < K ? nfull : K;
    uint64_t d = K;
    while (d < nfull && kl_extended(st, canon(h1[d - 1])))
        d++;
    return d;
}

static int kl_log_push(or_state *st, uint64_t ck)
{
    if (st->kl_log_n == st->kl_log_cap) {
        uint64_t cap = st->kl_log_cap ? 2 * st->kl_log_cap : 1024;
        uint64_t *a = (uint64_t *)realloc(st->kl_log, cap * sizeof(uint64_t));
        if (!a)
            return OR_ENOMEM;
        st->kl_log = a;
        st->kl_log_cap = cap;
    }
    st->kl_log[st->kl_log_n++] = ck;
    return OR_OK;
}

/* Turn the tree on with room for max_nodes extended prefixes (empty tree,
 * empty window), or off (max_nodes = 0). */
int or_keylen_enable(or_state *st, uint64_t max_nodes)
{
    if (!st)
        return OR_EINVAL;
    free(st->kl_ext);
    free(st->kl_log);
    st->kl_ext = NULL;
    st->kl_log = NULL;
    st->kl_n = st->kl_log_n = st->kl_log_cap = st->kl_win = 0;
    st->kl_on = max_nodes > 0;
    st->kl_max = max_nodes;
    if (max_nodes) {
        st->kl_ext = (uint64_t *)malloc(max_nodes * sizeof(uint64_t));
        if (!st->kl_ext) {
            st->kl_on = 0;
            return OR_ENOMEM;
        }
    }
    return OR_OK;
}

static int cmp_u64(const void *a, const void *b)
{
    uint64_t x = *(const uint64_t *)a, y = *(const uint64_t *)b;
    return x < y ? -1 : (x > y ? 1 : 0);
}

/* Close the window: the new tree is every prefix the window's requests
 * carry (depth >= K) that is hot, or extended and not cold, by its count
 * in the window; then start an empty window.  OR_EFULL (tree unchanged,
 * window still closed) if the new tree would hold more than max_nodes
 * extended prefixes. */
int or_keylen_window(or_state *st)
{
    if (!st || !st->kl_on)
        return OR_EINVAL;
    if (st->n_live == 0)
        return OR_ESTATE;
    const uint64_t W = st->kl_win, n = st->n_live;
    qsort(st->kl_log, st->kl_log_n, sizeof(uint64_t), cmp_u64);
    uint64_t *next = (uint64_t *)malloc((st->kl_log_n + st->kl_n + 1) * sizeof(uint64_t));
    if (!next)
        return OR_ENOMEM;
    uint64_t nn = 0;
    /* nodes seen in the window */
    for (uint64_t i = 0; i < st->kl_log_n;) {
        uint64_t j = i;
        while (j < st->kl_log_n && st->kl_log[j] == st->kl_log[i])
            j++;
        const uint64_t key = st->kl_log[i], c = j - i;
        if (kl_extended(st, key) ? c * n >= W : c * n > 2 * W)
            next[nn++] = key;
        i = j;
    }
    /* extended prefixes no request of the window carried: rho = 0 < 1/n,
     * unless the window is empty (no traffic, no change) */
    if (W == 0)
        for (uint64_t k = 0; k < st->kl_n; k++)
            next[nn++] = st->kl_ext[k];
    qsort(next, nn, sizeof(uint64_t), cmp_u64);
    uint64_t u = 0;
    for (uint64_t k = 0; k < nn; k++)
        if (u == 0 || next[k] != next[u - 1])
            next[u++] = next[k];
    int rc = OR_OK;
    if (u > st->kl_max) {
        rc = OR_EFULL;
    } else {
        memcpy(st->kl_ext, next, u * sizeof(uint64_t));
        st->kl_n = u;
    }
    free(next);
    st->kl_log_n = 0;
    st->kl_win = 0;
    return rc;
}

/* The extended prefixes, ascending (at most cap of them); *n gets the count. */
int or_keylen_export(const or_state *st, uint64_t *keys, uint64_t cap, uint64_t *n)
{
    if (!st || !n)
        return OR_EINVAL;
    for (uint64_t k = 0; k < st->kl_n && k < cap; k++)
        keys[k] = st->kl_ext[k];
    *n = st->kl_n;
    return OR_OK;
}

/* Route a batch in request order over a snapshot of the cached block sets,
 * applying each decision to the loads before the next request (scheduler
 * metadata is updated as requests are scheduled, Sec. A.3.2).
 * key[2n] ring keys, cand[2n] candidates, match[2n] cached blocks,
 * chosen[n], ttft[n], flags[n]; block_keys (optional) receives every full
 * block's f1 key, request-major; key_len (optional) each request's hashed
 * prefix length K_r in blocks.  With the hotness tree on, the ring keys hash
 * K_r blocks and each request's prefixes of depths K and more join the
 * current window. */
int or_route(or_state *st, const int32_t *tokens, const int64_t *off, uint64_t n,
             int64_t *loads, uint64_t *key, uint32_t *cand, uint32_t *match,
             uint32_t *chosen, int64_t *ttft, uint8_t *flags, uint64_t *block_keys,
             uint32_t *key_len)
{
    if (!st || (n && (!tokens || !off || !loads || !key || !cand || !match || !chosen ||
                      !ttft || !flags)))
        return OR_EINVAL;
    if (st->n_live == 0)
        return OR_ESTATE;
    const uint32_t B = st->cfg.block_size;
    uint64_t maxfull = 0;
    for (uint64_t r = 0; r < n; r++) {
        int64_t len = off[r + 1] - off[r];
        if (len < 0 || off[r] < 0)
            return OR_EINVAL;
        uint64_t nf = (uint64_t)len / B;
        if (nf > maxfull)
            maxfull = nf;
    }
    uint64_t *h1 = (uint64_t *)malloc((maxfull ? maxfull : 1) * sizeof(uint64_t));
    if (!h1)
        return OR_ENOMEM;
    uint64_t bk = 0;
    for (uint64_t r = 0; r < n; r++) {
        const int32_t *t = tokens + off[r];
        const int64_t len = off[r + 1] - off[r];
        const uint64_t nfull = or_chain(st, 0, t, len, h1);
        if (block_keys) {
            memcpy(block_keys + bk, h1, nfull * sizeof(uint64_t));
            bk += nfull;
        }
        const uint64_t kr = kl_key_len(st, h1, nfull);
        if (st->kl_on && nfull >= st->cfg.key_blocks)
            for (uint64_t d = st->cfg.key_blocks; d <= nfull; d++)
                if (kl_log_push(st, canon(h1[d - 1])) != OR_OK) {
                    free(h1);
                    return OR_ENOMEM;
                }
        if (key_len)
            key_len[r] = (uint32_t)kr;
        const uint64_t x1 = or_ring_key_at(st, 0, t, kr), x2 = or_ring_key_at(st, 1, t, kr);
        uint32_t c1, c2;
        uint8_t fl = or_candidates(st, x1, x2, &c1, &c2) ? 8 : 0;
        const uint64_t m1 = prefix_match(st, c1, h1, nfull);
        const uint64_t m2 = prefix_match(st, c2, h1, nfull);
        int64_t tt;
        const uint32_t ch = or_select(st, c1, c2, m1, m2, len, loads, &tt, &fl);
        loads[ch] += len - (int64_t)B * (int64_t)(ch == c1 ? m1 : m2);
        key[r] = x1; key[n + r] = x2;
        cand[r] = c1; cand[n + r] = c2;
        match[r] = (uint32_t)m1; match[n + r] = (uint32_t)m2;
        chosen[r] = ch; ttft[r] = tt; flags[r] = fl;
    }
    if (st->kl_on)
        st->kl_win += n;
    free(h1);
    return OR_OK;
}

/* ------------------------------------------------------------------------- */
/* Hotspot-aware rebalancing (Sec. 3.3, Eq. of the migration benefit;        */
/* Sec. A.1.2).                                                              */
/* ------------------------------------------------------------------------- */

typedef struct {
    int64_t benefit;
    uint64_t pos;     /* position in the source queue (head = 0) */
    uint64_t rec;     /* index into the record arrays             */
} or_cand;

static int cmp_cand(const void *pa, const void *pb)
{
    const or_cand *a = (const or_cand *)pa, *b = (const or_cand *)pb;
    if (a->benefit != b->benefit)
        return a->benefit > b->benefit ? -1 : 1; /* descending benefit */
    return a->pos < b->pos ? -1 : (a->pos > b->pos ? 1 : 0);
}

typedef struct {
    int64_t load;
    uint32_t id;
} or_src;

static int cmp_src(const void *pa, const void *pb)
{
    const or_src *a = (const or_src *)pa, *b = (const or_src *)pb;
    if (a->load != b->load)
        return a->load > b->load ? -1 : 1; /* heavier first */
    return a->id < b->id ? -1 : (a->id > b->id ? 1 : 0);
}

/* Largest estimated TTFT over the records still queued on an instance, each
 * record waiting behind the base work and the records ahead of it. */
static int64_t queue_max_ttft(const or_state *st, int64_t base_work, const uint32_t *unc,
                              const uint8_t *gone, uint64_t lo, uint64_t hi, int *any)
{
    int64_t ahead = base_work, mx = INT64_MIN;
    *any = 0;
    for (uint64_t q = lo; q < hi; q++) {
        if (gone[q - lo])
            continue;
        int64_t t = or_ttft(st, unc[q], ahead);
        if (t > mx)
            mx = t;
        ahead += unc[q];
        *any = 1;
    }
    return mx;
}

/* One single-round migration pass.  For every instance i the queue
 * [qoff[i], qoff[i+1]) lists its pending requests head first; record q
 * would cost unc_here[q] uncached tokens on i and unc_alt[q] on its
 * alternative candidate alt[q].  base_work[i] is work ahead of the queue.
 *
 *  - the TTFT of the record at queue position p on i waits behind base_work
 *    and the records ahead of it; i is overloaded if some queued TTFT
 *    exceeds the SLO (a long queue, Sec. 3.3), judged at pass start;
 *  - benefit of moving q from i to j: TTFT on i minus TTFT on j, both at pass
 *    start (Eq. of the migration benefit);
 *  - overloaded sources in order of load (heaviest first, ties by id);
 *    within a source, records with a positive benefit whose alternative is
 *    not overloaded, by descending benefit (ties: nearer the head first);
 *  - before each record: stop the source once every queued TTFT meets the
 *    SLO; the record moves only if its TTFT on j with j's current load is
 *    below the SLO (Sec. A.1.2); a move removes it from i's queue and adds
 *    unc_alt to j's load.  Moved records are not reconsidered.
 * loads_out[i] receives each instance's final load (base work plus its
 * queued uncached tokens plus received records).
 *
 * Decode-bottleneck correction (Sec. A.7), when prefill_interval is given:
 * an instance with a non-empty queue whose prefill interval (time since it
 * last completed a prefill) exceeds decode_threshold_us is taken to be
 * stalled in decode, and every TTFT estimated on it -- its queued records',
 * and a migrated record's as a target -- gets the interval added as the
 * decode-delay estimate D.  Loads are unchanged.  Intervals must lie in
 * [0, 2^40] and the threshold must not be negative. */
int or_rebalance(const or_state *st, const int64_t *qoff, const uint64_t *rec_id,
                 const uint32_t *unc_here, const uint32_t *alt, const uint32_t *unc_alt,
                 const int64_t *base_work, const int64_t *prefill_interval,
                 int64_t decode_threshold_us, int64_t *loads_out, uint64_t *mig_rec,
                 uint32_t *mig_from, uint32_t *mig_to, int64_t *mig_benefit,
                 int64_t *mig_ttft_to, uint64_t cap, uint64_t *count)
{
    if (!st || !qoff || !base_work || !loads_out || !count)
        return OR_EINVAL;
    const uint32_t S = st->cfg.max_slots;
    const int64_t slo = st->cfg.slo_us;
    for (uint32_t i = 0; i < S; i++)
        if (qoff[i + 1] < qoff[i] || qoff[i] < 0)
            return OR_EINVAL;
    const uint64_t Q = (uint64_t)qoff[S];
    for (uint64_t q = (uint64_t)qoff[0]; q < Q; q++)
        if (alt[q] >= S)
            return OR_EINVAL;
    if (decode_threshold_us < 0)
        return OR_EINVAL;
    if (prefill_interval)
        for (uint32_t i = 0; i < S; i++)
            if (prefill_interval[i] < 0 || prefill_interval[i] > ((int64_t)1 << 40))
                return OR_EINVAL;

    int64_t *L = (int64_t *)malloc(S * sizeof(int64_t));
    int64_t *maxT = (int64_t *)malloc(S * sizeof(int64_t));
    int64_t *D = (int64_t *)calloc(S, sizeof(int64_t));
    uint8_t *over = (uint8_t *)calloc(S, 1);
    or_src *src = (or_src *)malloc(S * sizeof(or_src));
    if (!L || !maxT || !D || !over || !src) {
        free(L); free(maxT); free(D); free(over); free(src);
        return OR_ENOMEM;
    }
    /* decode-delay estimate per instance (zero unless stalled in decode) */
    if (prefill_interval)
        for (uint32_t i = 0; i < S; i++)
            if (qoff[i + 1] > qoff[i] && prefill_interval[i] > decode_threshold_us)
                D[i] = prefill_interval[i];
    /* pass-start state */
    for (uint32_t i = 0; i < S; i++) {
        int64_t ahead = base_work[i], mx = INT64_MIN;
        for (int64_t q = qoff[i]; q < qoff[i + 1]; q++) {
            int64_t t = D[i] + or_ttft(st, unc_here[q], ahead);
            if (t > mx) mx = t;
            ahead += unc_here[q];
        }
        L[i] = ahead;
        maxT[i] = mx;
        over[i] = (qoff[i + 1] > qoff[i]) && mx > slo;
    }
    uint32_t nsrc = 0;
    for (uint32_t i = 0; i < S; i++)
        if (over[i]) {
            src[nsrc].load = L[i];
            src[nsrc].id = i;
            nsrc++;
        }
    qsort(src, nsrc, sizeof(or_src), cmp_src);

    int64_t *L0 = (int64_t *)malloc(S * sizeof(int64_t));
    if (!L0) {
        free(L); free(maxT); free(D); free(over); free(src);
        return OR_ENOMEM;
    }
    memcpy(L0, L, S * sizeof(int64_t));

    uint64_t nmig = 0;
    int rc = OR_OK;
    for (uint32_t si = 0; si < nsrc; si++) {
        const uint32_t i = src[si].id;
        const uint64_t lo = (uint64_t)qoff[i], hi = (uint64_t)qoff[i + 1];
        const uint64_t qlen = hi - lo;
        or_cand *c = (or_cand *)malloc((qlen ? qlen : 1) * sizeof(or_cand));
        uint8_t *gone = (uint8_t *)calloc(qlen ? qlen : 1, 1);
        if (!c || !gone) {
            free(c); free(gone);
            rc = OR_ENOMEM;
            break;
        }
        uint64_t nc = 0;
        int64_t ahead = base_work[i];
        for (uint64_t q = lo; q < hi; q++) {
            const int64_t ti = D[i] + or_ttft(st, unc_here[q], ahead);
            ahead += unc_here[q];
            const uint32_t j = alt[q];
            const int64_t tj = D[j] + or_ttft(st, unc_alt[q], L0[j]);
            const int64_t b = ti - tj;
            if (b > 0 && !over[j]) {
                c[nc].benefit = b;
                c[nc].pos = q - lo;
                c[nc].rec = q;
                nc++;
            }
        }
        qsort(c, nc, sizeof(or_cand), cmp_cand);
        int any;
        int64_t cur_max = queue_max_ttft(st, base_work[i], unc_here, gone, lo, hi, &any);
        for (uint64_t k = 0; k < nc; k++) {
            if (!any || D[i] + cur_max <= slo)
                break; /* every queued request meets the SLO */
            const uint64_t q = c[k].rec;
            const uint32_t j = alt[q];
            const int64_t tj = D[j] + or_ttft(st, unc_alt[q], L[j]);
            if (tj < slo) {
                gone[q - lo] = 1;
                L[i] -= unc_here[q];
                L[j] += unc_alt[q];
                if (nmig < cap) {
                    if (mig_rec) mig_rec[nmig] = rec_id ? rec_id[q] : q;
                    if (mig_from) mig_from[nmig] = i;
                    if (mig_to) mig_to[nmig] = j;
                    if (mig_benefit) mig_benefit[nmig] = c[k].benefit;
                    if (mig_ttft_to) mig_ttft_to[nmig] = tj;
                }
                nmig++;
                cur_max = queue_max_ttft(st, base_work[i], unc_here, gone, lo, hi, &any);
            }
        }
        free(c);
        free(gone);
    }
    memcpy(loads_out, L, S * sizeof(int64_t));
    *count = nmig;
    free(L); free(L0); free(maxT); free(D); free(over); free(src);
    if (rc == OR_OK && nmig > cap)
        rc = OR_EFULL;
    return rc;
}

/* ------------------------------------------------------------------------- */
/* Dual-hash-ring scaling (Sec. 3.4; Sec. A.1.3).                            */
/* ------------------------------------------------------------------------- */

/* Add instances add[0..n_add) and remove rm[0..n_rm): both rings are rebuilt
 * for the new live set.  For every ring key keys[s*n + k] (ring s = 0, 1) the
 * owner before and after is reported; moved[s] counts keys whose owner
 * changed, violations counts moves that neither leave a removed instance nor
 * land on an added one (consistent hashing says there are none).  Removed
 * instances lose their cached sets; added ones start empty. */
int or_scale(or_state *st, const uint32_t *add, uint32_t n_add, const uint32_t *rm, uint32_t n_rm,
             const uint64_t *keys, uint64_t n, uint32_t *old_owner, uint32_t *new_owner,
             uint64_t *moved, uint64_t *violations)
{
    if (!st || (n_add && !add) || (n_rm && !rm) || (n && (!keys || !old_owner || !new_owner)) ||
        !moved || !violations)
        return OR_EINVAL;
    if (st->n_live == 0)
        return OR_ESTATE;
    const uint32_t S = st->cfg.max_slots;
    uint8_t *is_add = (uint8_t *)calloc(S, 1), *is_rm = (uint8_t *)calloc(S, 1);
    if (!is_add || !is_rm) {
        free(is_add); free(is_rm);
        return OR_ENOMEM;
    }
    int bad = 0;
    for (uint32_t k = 0; k < n_add; k++) {
        if (add[k] >= S || st->live[add[k]] || is_add[add[k]]) bad = 1;
        else is_add[add[k]] = 1;
    }
    for (uint32_t k = 0; k < n_rm; k++) {
        if (rm[k] >= S || !st->live[rm[k]] || is_rm[rm[k]]) bad = 1;
        else is_rm[rm[k]] = 1;
    }
    if (!bad && st->n_live - n_rm + n_add == 0)
        bad = 1;
    if (bad) {
        free(is_add); free(is_rm);
        return OR_EINVAL;
    }
    for (uint64_t k = 0; k < 2 * n; k++)
        old_owner[k] = ring_owner(st, (int)(k / (n ? n : 1)), keys[k]);
    for (uint32_t id = 0; id < S; id++) {
        if (is_rm[id] || is_add[id]) {
            st->live[id] = is_add[id] ? 1 : 0;
            free(st->set[id]); st->set[id] = NULL; st->set_len[id] = 0;
            /* the saved-key record of an emptied cache goes with it */
            free(st->lru_key[id]); st->lru_key[id] = NULL;
            free(st->lru_t[id]); st->lru_t[id] = NULL;
            st->lru_len[id] = 0;
        }
    }
    st->n_live = st->n_live - n_rm + n_add;
    int rc = rebuild_rings(st);
    if (rc != OR_OK) {
        free(is_add); free(is_rm);
        return rc;
    }
    moved[0] = moved[1] = 0;
    *violations = 0;
    for (uint64_t k = 0; k < 2 * n; k++) {
        const int s = (int)(k / n);
        new_owner[k] = ring_owner(st, s, keys[k]);
        if (new_owner[k] != old_owner[k]) {
            moved[s]++;
            if (!is_rm[old_owner[k]] && !is_add[new_owner[k]])
                (*violations)++;
        }
    }
    free(is_add); free(is_rm);
    return OR_OK;
}

uint32_t or_n_live(const or_state *st) { return st ? st->n_live : 0; }
