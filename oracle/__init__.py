"""Plain CPU oracle of the plan search (test infrastructure only)."""
