/*
 * cpu_manager.c -- a multi-threaded memory manager on the host: the free-list
 * compaction (completion recycling) and page allocation of the paged cache,
 * run over all tables by a pool of worker threads.  This is the on-CPU
 * alternative the paper measures its on-GPU parallel compaction against
 * (Sec. 7, memory management overhead); it is a comparison baseline for the
 * benchmark, not part of the library and not the test oracle.
 *
 * State and results are those of the library's diffkv_compact_free_list and
 * diffkv_alloc_pages on the same host arrays: tables ascending, released IDs
 * in ascending slot order written at the end pointer, kept high IDs packed to
 * the left and low IDs to the right in their order, vacated slots -1; new IDs
 * taken from the start pointer, high pages left to right then low pages right
 * to left, table by table; all-or-nothing allocation.
 *
 * Parallel structure (both operations): every worker counts its contiguous
 * range of tables, one worker forms the exclusive prefix over the workers'
 * totals, then every worker writes its tables' ring region and rows.  Workers
 * wait on a shared barrier between the phases; the pool is created once.
 */
#define _POSIX_C_SOURCE 200809L
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int32_t* table;     /* [num_tables][p_max], -1 = empty */
    int32_t* pages;     /* [num_tables][2] */
    int32_t* len;       /* [num_tables][2] */
    int32_t* ring;      /* [num_pages] */
    int64_t* ring_ptr;  /* [2] {head, tail} */
    uint32_t* status;   /* [1] sticky bits: 1 out of pages, 2 table overflow */
    int64_t num_pages;
    int32_t num_tables;
    int32_t p_max;
    int32_t tokens_per_page[2];
} cm_state;

enum { CM_OP_QUIT = 0, CM_OP_COMPACT = 1, CM_OP_ALLOC = 2 };

typedef struct cm_pool {
    int n;
    pthread_t* th;
    pthread_barrier_t go, sync, done;
    int op;
    cm_state* st;
    const void* arg;     /* release [T][p_max] or demand [T][2] */
    int64_t* part;       /* per worker: count of its tables, then its ring offset */
    uint32_t* bad;       /* per worker: allocation check bits */
    int64_t total;
    int refused;
} cm_pool;

typedef struct {
    cm_pool* pool;
    int w;
} cm_worker;

static void range_of(const cm_pool* p, int w, int* t0, int* t1)
{
    int64_t T = p->st->num_tables;
    *t0 = (int)(T * w / p->n);
    *t1 = (int)(T * (w + 1) / p->n);
}

/* after the counting phase: exclusive prefix over the workers, by worker 0 */
static void prefix(cm_pool* p)
{
    int64_t run = 0;
    for (int i = 0; i < p->n; i++) {
        int64_t c = p->part[i];
        p->part[i] = run;
        run += c;
    }
    p->total = run;
}

static void compact_worker(cm_pool* p, int w)
{
    cm_state* s = p->st;
    const uint8_t* release = (const uint8_t*)p->arg;
    const int P = s->p_max;
    int t0, t1;
    range_of(p, w, &t0, &t1);
    int64_t cnt = 0;
    for (int t = t0; t < t1; t++) {
        const uint8_t* rel = release + (int64_t)t * P;
        int ph = s->pages[2 * t], pl = s->pages[2 * t + 1];
        for (int k = 0; k < ph; k++) cnt += rel[k] != 0;
        for (int k = P - pl; k < P; k++) cnt += rel[k] != 0;
    }
    p->part[w] = cnt;
    pthread_barrier_wait(&p->sync);
    if (w == 0) prefix(p);
    pthread_barrier_wait(&p->sync);
    int64_t tail = s->ring_ptr[1] + p->part[w];
    int32_t* keep = (int32_t*)malloc(sizeof(int32_t) * (size_t)P);
    for (int t = t0; t < t1; t++) {
        int32_t* row = s->table + (int64_t)t * P;
        const uint8_t* rel = release + (int64_t)t * P;
        int ph = s->pages[2 * t], pl = s->pages[2 * t + 1];
        int lens[2] = {s->len[2 * t], s->len[2 * t + 1]};
        int dropped[2] = {0, 0};
        for (int slot = 0; slot < P; slot++) {
            int sec, k;
            if (slot < ph) { sec = 0; k = slot; }
            else if (slot >= P - pl) { sec = 1; k = P - 1 - slot; }
            else continue;
            if (!rel[slot]) continue;
            s->ring[tail % s->num_pages] = row[slot];
            tail++;
            int T = s->tokens_per_page[sec];
            int fill = lens[sec] - k * T;
            dropped[sec] += fill < 0 ? 0 : (fill > T ? T : fill);
        }
        int nk = 0;
        for (int k = 0; k < ph; k++)
            if (!rel[k]) keep[nk++] = row[k];
        for (int k = 0; k < ph; k++) row[k] = k < nk ? keep[k] : -1;
        s->pages[2 * t] = nk;
        nk = 0;
        for (int k = 0; k < pl; k++)
            if (!rel[P - 1 - k]) keep[nk++] = row[P - 1 - k];
        for (int k = 0; k < pl; k++) row[P - 1 - k] = k < nk ? keep[k] : -1;
        s->pages[2 * t + 1] = nk;
        s->len[2 * t] -= dropped[0];
        s->len[2 * t + 1] -= dropped[1];
    }
    free(keep);
}

static void alloc_worker(cm_pool* p, int w)
{
    cm_state* s = p->st;
    const int32_t* demand = (const int32_t*)p->arg;
    const int P = s->p_max;
    int t0, t1;
    range_of(p, w, &t0, &t1);
    int64_t cnt = 0;
    uint32_t bad = 0;
    for (int t = t0; t < t1; t++) {
        int64_t nh = demand[2 * t], nl = demand[2 * t + 1];
        cnt += nh + nl;
        if ((int64_t)s->pages[2 * t] + nh + s->pages[2 * t + 1] + nl > P) bad |= 2u;
    }
    p->part[w] = cnt;
    p->bad[w] = bad;
    pthread_barrier_wait(&p->sync);
    if (w == 0) {
        prefix(p);
        uint32_t all = 0;
        for (int i = 0; i < p->n; i++) all |= p->bad[i];
        if (p->total > s->ring_ptr[1] - s->ring_ptr[0]) all |= 1u;
        p->refused = all != 0;
        if (all) *s->status |= all;
    }
    pthread_barrier_wait(&p->sync);
    if (p->refused) return;
    int64_t head = s->ring_ptr[0] + p->part[w];
    for (int t = t0; t < t1; t++) {
        int32_t* row = s->table + (int64_t)t * P;
        for (int i = 0; i < demand[2 * t]; i++) row[s->pages[2 * t]++] = s->ring[head++ % s->num_pages];
        for (int i = 0; i < demand[2 * t + 1]; i++)
            row[P - 1 - s->pages[2 * t + 1]++] = s->ring[head++ % s->num_pages];
    }
}

static void* worker_main(void* a)
{
    cm_worker* me = (cm_worker*)a;
    cm_pool* p = me->pool;
    for (;;) {
        pthread_barrier_wait(&p->go);
        if (p->op == CM_OP_QUIT) break;
        if (p->op == CM_OP_COMPACT) compact_worker(p, me->w);
        else alloc_worker(p, me->w);
        pthread_barrier_wait(&p->done);
    }
    free(me);
    return NULL;
}

cm_pool* cm_pool_create(int nthreads)
{
    if (nthreads < 1) return NULL;
    cm_pool* p = (cm_pool*)calloc(1, sizeof(cm_pool));
    p->n = nthreads;
    p->th = (pthread_t*)calloc((size_t)nthreads, sizeof(pthread_t));
    p->part = (int64_t*)calloc((size_t)nthreads, sizeof(int64_t));
    p->bad = (uint32_t*)calloc((size_t)nthreads, sizeof(uint32_t));
    pthread_barrier_init(&p->go, NULL, (unsigned)nthreads + 1);
    pthread_barrier_init(&p->done, NULL, (unsigned)nthreads + 1);
    pthread_barrier_init(&p->sync, NULL, (unsigned)nthreads);
    for (int i = 0; i < nthreads; i++) {
        cm_worker* me = (cm_worker*)malloc(sizeof(cm_worker));
        me->pool = p;
        me->w = i;
        pthread_create(&p->th[i], NULL, worker_main, me);
    }
    return p;
}

static void run(cm_pool* p, int op, cm_state* s, const void* arg)
{
    p->op = op;
    p->st = s;
    p->arg = arg;
    pthread_barrier_wait(&p->go);
    pthread_barrier_wait(&p->done);
}

/* Completion recycling: every live slot whose release byte is nonzero. */
void cm_compact(cm_pool* p, cm_state* s, const uint8_t* release)
{
    run(p, CM_OP_COMPACT, s, release);
    s->ring_ptr[1] += p->total;
}

/* Page allocation; returns 0, or 1 when refused (status bits raised). */
int cm_alloc(cm_pool* p, cm_state* s, const int32_t* demand)
{
    run(p, CM_OP_ALLOC, s, demand);
    if (p->refused) return 1;
    s->ring_ptr[0] += p->total;
    return 0;
}

void cm_pool_destroy(cm_pool* p)
{
    if (!p) return;
    p->op = CM_OP_QUIT;
    pthread_barrier_wait(&p->go);
    for (int i = 0; i < p->n; i++) pthread_join(p->th[i], NULL);
    pthread_barrier_destroy(&p->go);
    pthread_barrier_destroy(&p->done);
    pthread_barrier_destroy(&p->sync);
    free(p->th);
    free(p->part);
    free(p->bad);
    free(p);
}
