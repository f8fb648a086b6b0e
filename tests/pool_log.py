"""Replays a pool's event record (fo_queues_log_read) through the oracle's
Task Scheduler and checks every event against it: admissions and refusals,
sequence numbers, the device, sequence number and slot of every pick, the
model served at every aggregation with its staleness and skip decision, and
leave / rejoin transitions.  A record that replays cleanly is a valid
interleaving of put() and get() (Alg. 2, Alg. 3) under the flow control of
Sec. 3.4.1; the replay also returns the picks and the applied aggregations in
order, from which the trained and aggregated models can be rebuilt."""
from oracle.scheduler import TaskScheduler

EV_PUSH, EV_MODEL, EV_PICK, EV_RELEASE, EV_AGG, EV_LEAVE, EV_JOIN = range(1, 8)


def replay(log, K, n_slots, policy="counter", max_delay=None):
    sch = TaskScheduler(K, n_slots, policy=policy)
    picks, aggs, models = [], [], {}
    model_count = [0] * K
    for i, (typ, k, a, b) in enumerate(log.tolist()):
        where = (i, typ, k, a, b)
        if typ == EV_PUSH:
            ok, seq, _ = sch.put_act(k)
            assert (int(ok), seq if ok else -1) == (a, b), where
        elif typ == EV_MODEL:
            sch.put_model(k, a)
            models.setdefault(k, []).append((model_count[k], a))
            model_count[k] += 1
        elif typ == EV_PICK:
            r = sch.get()
            assert r == ("act", k, a, b), (where, r)
            picks.append((k, a))
        elif typ == EV_RELEASE:
            sch.release()
        elif typ == EV_AGG:
            r = sch.get()
            assert r is not None and r[0] == "model" and r[1] == k, (where, r)
            applied, s = sch.aggregate_version(r[2], max_delay)
            assert (int(applied), s) == (a, b), where
            r_index = models[k].pop(0)[0]  # the device's r-th model message
            aggs.append((k, r_index, s, applied))
        elif typ == EV_LEAVE:
            sch.set_active(k, False)
        elif typ == EV_JOIN:
            if a == 1:
                assert sch.add_device() == k, where
            else:
                sch.set_active(k, True)
        else:
            raise AssertionError(f"unknown event {where}")
    return sch, picks, aggs
