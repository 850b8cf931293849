"""The oracle's sender plan and packing (Sec. 4.1.2), pinned by rebuilding every payload
from the plan alone: cache hits from the bytes the server holds (keyed by content),
batch repeats from the earlier block's bytes, misses from the packed buffer."""

import numpy as np

import oracle


def test_plan_pack_rebuilds_payloads():
    rng = np.random.default_rng(81)
    block = 4096
    for trial in range(10):
        pool = [rng.bytes(block) for _ in range(6)]
        server_has = {pool[i] for i in range(3)}
        payloads = []
        for _ in range(8):
            parts = [pool[int(i)] for i in rng.integers(0, 6, int(rng.integers(0, 5)))]
            payloads.append(np.frombuffer(b"".join(parts) + rng.bytes(int(rng.integers(0, 3000))), np.uint8))
        table = oracle.Table()
        for b in server_has:
            d, _ = oracle.payload_digests(np.frombuffer(b, np.uint8), block)
            table.insert(d, np.array([0], np.uint64))
        res = oracle.run(payloads, block, table)
        lens = [p.size for p in payloads]
        rec, tot = oracle.send_plan(lens, block, res["digests"], res["status"], res["ref"])
        packed = oracle.pack_misses(payloads, rec, int(tot[3]))
        by_digest = {}
        for b in server_has:
            by_digest[int(oracle.payload_digests(np.frombuffer(b, np.uint8), block)[0][0])] = b
        rebuilt = [bytearray(n) for n in lens]
        for r in rec:  # in batch order, so a repeat's source is already rebuilt
            o, ln, s = int(r["offset"]), int(r["length"]), int(r["payload"])
            if r["kind"] == oracle.MISS:
                src = packed[int(r["ident"]):int(r["ident"]) + ln].tobytes()
            elif r["kind"] == oracle.HIT_CACHE:
                src = by_digest[int(r["ident"])]
            else:
                e = rec[int(r["ident"])]
                src = bytes(rebuilt[int(e["payload"])][int(e["offset"]):int(e["offset"]) + ln])
            rebuilt[s][o:o + ln] = src
        assert all(bytes(rb) == p.tobytes() for rb, p in zip(rebuilt, payloads)), trial
        assert int(tot[0] + tot[1] + tot[2]) == rec.size
        assert all(int(r["ident"]) % 16 == 0 for r in rec[rec["kind"] == oracle.MISS])
