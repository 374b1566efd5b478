"""MI355X batched backward dataflow enumeration (Dirigo's per-location
back-projection, Sec. 3.4 of the Output-Space Hypothesis paper).

Import ``paper_2609_19611_amd.binding`` for the C-ABI library and
``paper_2609_19611_amd.workloads`` for the seeded synthetic inputs.
"""
