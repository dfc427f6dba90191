"""CPU oracle for the PVS dense channel and exact adaptive hybrid retrieval.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import anything from this package; the
product path (``libeahr.so`` and its binding) never does.

Every function here is a plain, slow transcription of a definition from the
paper "Exact Adaptive Hybrid Retrieval Without Fixed Top-L Cutoffs":

* :mod:`oracle.pvs`     PVS quantisation and score intervals (Sec. 2.3.1, App. A.1)
* :mod:`oracle.dense`   exact dense ranking (Sec. 2.1 complete ranked lists)
* :mod:`oracle.sparse`  brute-force sparse scores and ranking (Sec. 2.3.2, App. A.2)
* :mod:`oracle.rrf`     complete-list weighted RRF Top-K (Sec. 2.1)
* :mod:`oracle.certify` ordered certification from revealed prefixes (Sec. 2.2)

It shares no code with the HIP path; both read inputs only from
``paper_2608_07152_amd.datagen`` (which holds none of the method's arithmetic).
Parity status of each function is stated in its module docstring.
"""
