"""VGGT-Prime routed global attention on MI355X (gfx950).

The binding to the HIP library is in ``paper_2609_23733_amd.vp``; importing
the package itself loads nothing, so the seeded input generators
(``paper_2609_23733_amd.synth``) can be used without a GPU.
"""
