"""Oracle sessions in worker processes.

TEST INFRASTRUCTURE ONLY (like the rest of this package): the parity tests
and the benchmark's CPU-baseline leg use it to run the sessions of a batch
side by side on the host's cores.  Each worker is a fresh Python process
(a child interpreter that connects back over a Unix socket, so a caller
that uses the GPU hands nothing of it on) with one BLAS thread, holding some of the batch's
``Session`` objects; a step sends every worker its sessions' inputs and
gathers their records.  Nothing here changes what a session computes.
"""
from __future__ import annotations

import os
import secrets
import subprocess
import sys
from multiprocessing.connection import Client, Listener
from typing import Dict, List, Optional, Tuple

_ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

_ONE_THREAD = {k: "1" for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS",
                                "BLIS_NUM_THREADS", "NUMEXPR_NUM_THREADS")}


def host_cores() -> int:
    """Cores this process may run on."""
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def _worker_main(address: str, key_hex: str) -> None:
    """Entry of a worker process: connect back to the pool and serve."""
    _serve(Client(address, family="AF_UNIX", authkey=bytes.fromhex(key_hex)))


def _serve(conn) -> None:
    from .memdecay import Session
    sessions: Dict[int, Session] = {}
    while True:
        msg = conn.recv()
        kind = msg[0]
        if kind == "add":
            _, s, kwargs, keys_bits = msg
            sessions[s] = Session(keys_bits=keys_bits, **kwargs)
            conn.send(None)
        elif kind == "step":
            out = {}
            for s, (q, nk, reg) in msg[1].items():
                out[s] = sessions[s].step(q, nk, reg)
            conn.send(out)
        elif kind == "close":
            conn.send(None)
            return


class SessionPool:
    """Sessions spread over ``workers`` processes; a session goes to the
    worker with the fewest tokens so far (``weight``)."""

    def __init__(self, workers: Optional[int] = None):
        n = max(1, min(workers or host_cores(), 64))
        key = secrets.token_bytes(16)
        listener = Listener(family="AF_UNIX", authkey=key)
        env = dict(os.environ, **_ONE_THREAD)
        code = (f"import sys; sys.path.insert(0, {_ROOT!r}); from oracle.pool import _worker_main; "
                f"_worker_main({listener.address!r}, {key.hex()!r})")
        self._procs = [subprocess.Popen([sys.executable, "-c", code], env=env, cwd=_ROOT) for _ in range(n)]
        self._conns = [listener.accept() for _ in range(n)]
        listener.close()
        self.workers = n
        self._load = [0] * n
        self._home: Dict[int, int] = {}

    def add(self, s: int, kwargs: dict, keys_bits, weight: int) -> None:
        """Create session s in the least loaded worker (keys_bits: the
        session's prompt keys, bf16 bits [n][L][Hkv][d])."""
        i = min(range(self.workers), key=lambda j: self._load[j])
        self._load[i] += max(int(weight), 1)
        self._home[s] = i
        self._conns[i].send(("add", s, kwargs, keys_bits))
        self._conns[i].recv()

    def step(self, inputs: Dict[int, Tuple]) -> Dict[int, object]:
        """One step of every given session: inputs[s] = (q, new_key_bits,
        new_region); returns {s: StepRecord}, all workers running at once."""
        per: List[dict] = [dict() for _ in range(self.workers)]
        for s, inp in inputs.items():
            per[self._home[s]][s] = inp
        busy = [i for i in range(self.workers) if per[i]]
        for i in busy:
            self._conns[i].send(("step", per[i]))
        out: Dict[int, object] = {}
        for i in busy:
            out.update(self._conns[i].recv())
        return out

    def close(self) -> None:
        for c in self._conns:
            try:
                c.send(("close",))
                c.recv()
            except (OSError, EOFError):
                pass
        for p in self._procs:
            try:
                p.wait(timeout=10)
            except subprocess.TimeoutExpired:
                p.kill()
                p.wait()
        self._conns, self._procs = [], []
