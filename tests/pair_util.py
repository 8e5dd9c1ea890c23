"""The pair schedule (lvsa.h) by its definition, for tests."""


def expected_pairs(row_ptr, col_idx, entry=None):
    """The pair schedule by its definition: row p is the union of CSR rows
    2p and 2p+1, each key block tagged with the rows that hold it (block
    form), or with their entry words' patterns (token-exact form)."""
    nb = len(row_ptr) - 1
    ptr, words, exact = [0], [], []
    for p in range(-(-nb // 2)):
        rows = [2 * p] + ([2 * p + 1] if 2 * p + 1 < nb else [])
        held = [dict((int(col_idx[i]), i) for i in range(row_ptr[r], row_ptr[r + 1]))
                for r in rows] + [{}]
        for kb in sorted(set(held[0]) | set(held[1])):
            words.append(kb | (kb in held[0]) << 30 | (kb in held[1]) << 31)
            if entry is not None:
                e = [int(entry[h[kb]]) if kb in h else 0 for h in held[:2]]
                base = (e[0] or e[1]) & 0xFFFFFF
                exact.append(base | ((e[0] >> 24) & 0xF) << 24 | ((e[1] >> 24) & 0xF) << 28)
        ptr.append(len(words))
    return ptr, words, exact
